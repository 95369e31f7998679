// Internal interface between the C ABI (abi.cpp) and the HIP kernels.
// Every launcher enqueues on `stream` and returns the launch status.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace l4d {

// Rows of a token-major activation that may be split between this rank's own
// sequence-parallel rows and the rows the all-gather brings from the peers.
// Logical row m (0 <= m < b*s_c) lives at own + (...)*ld when its in-sequence
// index i = m % s_c falls in [r*s_sp, (r+1)*s_sp), else in peer.
// With t == 1 (or peer == nullptr) it is simply base + m*ld.
struct RowSrc {
  const uint16_t* own;
  const uint16_t* peer;
  int64_t ld;     // elements between consecutive rows
  int32_t s_c;    // rows per batch element of the gathered view
  int32_t s_sp;   // own rows per batch element
  int32_t r;      // own slot
  int32_t t;      // slots (1 = not split)

  __host__ __device__ static RowSrc plain(const void* p, int64_t ld) {
    return RowSrc{static_cast<const uint16_t*>(p), nullptr, ld, 1, 1, 0, 1};
  }
  // Row m as (index into own) or (index into peer) | 0x80000000; 32-bit arithmetic
  // (row counts are validated below 2^30 on the host).
  __device__ __forceinline__ uint32_t row_index(int64_t m64) const {
    const int32_t m = static_cast<int32_t>(m64);
    if (t == 1) return static_cast<uint32_t>(m);
    const int32_t bi = m / s_c;
    const int32_t i = m - bi * s_c;
    const int32_t lo = r * s_sp;
    if (i >= lo && i < lo + s_sp) return static_cast<uint32_t>(bi * s_sp + (i - lo));
    const int32_t pi = i < lo ? i : i - s_sp;
    return static_cast<uint32_t>(bi * (t - 1) * s_sp + pi) | 0x80000000u;
  }
  __device__ __forceinline__ const uint16_t* row(int64_t m) const {
    const uint32_t o = row_index(m);
    return ((o & 0x80000000u) ? peer : own) + static_cast<int64_t>(o & 0x7fffffffu) * ld;
  }
};

// One GEMM operand.  "kc" (k-contiguous): element (x, k) at src.row(x)[k].
// "mn" (mn-contiguous): element (x, k) at src.row(k)[x].
// split: (k-contiguous B only) tile rows [0,128) of N-tile j come from rows
// j*128 + [0,128) and tile rows [128,256) from split_off + j*128 + [0,128);
// rows with j*128 + i >= split_rows are zero.  Used to interleave the gate
// and up halves of a fused [gate; up] weight so one tile holds both.
struct Operand {
  RowSrc src;
  int32_t rows;        // extent of the non-k index (M for A, N for B) in storage
  int32_t split_rows;  // 0 = no split
  int64_t split_off;
};

enum class Layout { KC, MN };

// ---------------------------------------------------------------- epilogues
// Every GEMM hands its fp32 tile to one of these, as 8-column vectors.

enum class EpiKind {
  StoreBF16,    // C (bf16) = acc, row-major with ldc
  StoreF32,     // C (f32) = acc, row-major with ldc
  AccF32,       // C (f32) += acc
  QkvRope,      // split [Q|K|V] columns, RoPE on Q and K, bf16
  ResidualSP,   // own rows: bf16 or fp32 (acc + resid + receipt); peer rows: bf16(acc) -> send buffer
  SwiGLUFwd,    // gate/up tile pairs -> G, U, act, prod (bf16)
  SwiGLUBwd     // acc = d(prod) -> dG, dU from the stashed G, U, act
};

struct EpiParams {
  EpiKind kind;
  void* c;              // StoreBF16 / AccF32 output
  int64_t ldc;
  // QkvRope
  uint16_t *q, *k, *v;
  int32_t nq, nk;       // columns of Q and of K (= of V)
  const float2* rope;   // [tokens_per_batch][d_h/2] (cos, sin) by local row
  int32_t d_h;
  // ResidualSP (rows in the gathered view; own rows mapped like RowSrc)
  uint16_t* own_out;    // [b*s_sp][ldc]
  float* own_out_f32;   // when set, the own rows are stored here in fp32 instead
  const uint16_t* resid;    // may be null
  const uint16_t* receipt;  // may be null
  uint16_t* send;       // [b*(t-1)*s_sp][ldc]
  int32_t s_c, s_sp, r, t;
  // SwiGLUFwd / SwiGLUBwd: [tokens][f] tensors, f = split_rows of B
  uint16_t *g_out, *u_out, *act_out, *prod_out;
  const uint16_t *g_in, *u_in, *act_in;
  uint16_t* dgu;        // [tokens][2f] : dG columns [0,f), dU columns [f,2f)
  int32_t f;
};

struct GemmParams {
  int32_t M, N, K;
  Operand A, B;
  EpiParams epi;
  // AccF32 and StoreBF16 only: the K range is cut into k_splits equal parts
  // (0 or 1 = none).  AccF32: part 0 accumulates into C; part s > 0 stores its
  // fp32 sum to partial + (s - 1) M N (row-major, ld N), which
  // gemm_split_reduce then adds to C in order s = 1, 2, ...  StoreBF16: part s
  // stores to partial + s M N and gemm_split_store writes bf16(sum) to C.
  int32_t k_splits;
  float* partial;
};

hipError_t gemm(const GemmParams& p, Layout la, Layout lb, hipStream_t stream);
// Parts the K range of an fp32-accumulate GEMM is cut into when one tile per
// workgroup would leave much of the chip idle (1 = no split).
int gemm_ksplits(int64_t M, int64_t N, int64_t K, bool acc_f32);
// C[m][n] += sum over s of partial[s][m][n], s = 0 .. splits - 2, in that order.
hipError_t gemm_split_reduce(float* c, int64_t ldc, const float* partial, int64_t M, int64_t N, int32_t splits,
                             hipStream_t stream);
// C (bf16) = sum over s of partial[s], s = 0 .. splits - 1, in that order
// (splits = 1: the fp32 partial rounded to bf16).
hipError_t gemm_split_store(uint16_t* c, int64_t ldc, const float* partial, int64_t M, int64_t N, int32_t splits,
                            hipStream_t stream);

// ---------------------------------------------------------------- row-wise kernels

// y = bf16(gain * x * rsqrt(mean(x^2) + eps)), one row of h per wave; x is
// also copied to x_copy when that is not null.
hipError_t rmsnorm_fwd(const uint16_t* x, const uint16_t* gain, uint16_t* y, int64_t rows,
                       int32_t h, float eps, hipStream_t stream, uint16_t* x_copy = nullptr);
// RMSNorm backward: dx = dres + d rmsnorm/dx . dy, stored bf16 (and fp32 when
// dx_f32 is set);  partial[blk][h] = sum over the block's rows of dy*xhat.
// dy is bf16 (dy) or fp32 (dy_f32); dres is absent, bf16 or fp32.  Forms:
// (bf16 dy, no dres), (fp32 dy, bf16 dres, fp32 copy), (fp32 dy, fp32 dres).
struct NormBwdIo {
  const uint16_t* dy;
  const float* dy_f32;
  const uint16_t* dres;
  const float* dres_f32;
  uint16_t* dx;
  float* dx_f32;
};
hipError_t rmsnorm_bwd(const uint16_t* x, const uint16_t* gain, const NormBwdIo& io, float* partial,
                       int32_t n_partial, int64_t rows, int32_t h, float eps, hipStream_t stream);
// out[j] += sum_i partial[i][j] in a fixed order; with more than 256 rows partial
// is overwritten (used as scratch).
hipError_t reduce_rows_add(float* partial, int32_t n_partial, int32_t h, float* out, hipStream_t stream);
int32_t rmsnorm_bwd_partials(int64_t rows);

// cos/sin table for RoPE: tab[i][j] = (cos, sin)(pos_i * base^(-2j/d_h)), computed in fp64.
struct ChunkMap {          // local row -> global position
  int32_t n_chunks;        // 1 or 2
  int32_t chunk_len;
  int32_t chunk_id[2];
};
hipError_t rope_table(float2* tab, ChunkMap map, int32_t rows, int32_t d_h, float base,
                      hipStream_t stream);

// ---------------------------------------------------------------- attention

// A run of keys with consecutive global positions.
struct KvSeg {
  const uint16_t* k;   // token 0 of the run: [tokens][ld], head hk at column hk*d_h
  const uint16_t* v;
  int64_t ld, bstride;     // row and batch strides of k, v, rk, rv (elements)
  uint16_t* dk;        // backward outputs, may be null in the forward
  uint16_t* dv;
  int64_t d_ld, d_bstride; // row and batch strides of dk, dv
  const uint16_t* rk;  // receipts added before storing dk/dv (null = none)
  const uint16_t* rv;
  int32_t n;           // tokens
  int32_t pos0;        // global position of token 0
  int32_t rope;        // 1: apply the inverse RoPE to dk (local keys)
  int32_t rope_row0;   // row of token 0 in the RoPE table
};
constexpr int kMaxSeg = 8;

struct AttnParams {
  int32_t b, a_t, k_t, d_h;
  int32_t n_q;                 // local query rows per batch element
  int64_t q_ld, q_bstride;     // strides of q, o, dout (elements)
  const uint16_t* q;           // [b][n_q][a_t*d_h]
  uint16_t* o;                 // ctx, same layout
  float* lse;                  // [b][a_t][n_q], natural log
  ChunkMap qmap;               // local query row -> global position
  int32_t n_seg;
  KvSeg seg[kMaxSeg];
  float scale;                 // 1/sqrt(d_h)
  // backward
  const uint16_t* dout;        // dctx
  float* delta;                // [b][a_t][n_q]
  uint16_t* dq;                // [b][n_q][dq_ld] at column h*d_h, inverse RoPE applied
  int64_t dq_ld;
  const float2* rope;          // table used by the inverse RoPE
  // dK/dV split over query-head slices (n_split > 1): fp32 partials
  // [n_split][b][total_keys][k_t][d_h] for dK, then the same for dV at +partial_half
  int32_t n_split;
  int32_t total_keys;          // keys over all segments
  int32_t seg_key0[kMaxSeg];   // index of each segment's first key among them
  float* dkv_partial;
  int64_t partial_half;
  // dK/dV: the 128-key blocks in the order the grid dispatches them (heaviest
  // first; filled by attn_bwd when there are at most kMaxKeyBlocks, else n_order = 0
  // and blocks go in key order)
  int32_t n_order;
  uint16_t kb_order[512];
};
constexpr int kMaxKeyBlocks = 512;

// Number of query-head slices the dK/dV pass uses for this shape (1 = none).
int attn_bwd_splits(const AttnParams& p);
hipError_t attn_fwd(const AttnParams& p, hipStream_t stream);
// part 2: dQ, and delta = rowsum(dO * O) for part 1; 1: dK, dV (after part 2);
// 3: the sum of the query-head slices of dK, dV when n_split > 1 (nothing otherwise).
hipError_t attn_bwd(const AttnParams& p, int part, hipStream_t stream);

// ---------------------------------------------------------------- cross-entropy

hipError_t xent_rows(const uint16_t* logits, int64_t n, int32_t v_t, int64_t v0,
                     const int64_t* targets, const float* peer_lse, const float* peer_z,
                     float grad_scale, float* loss, uint16_t* dlogits, hipStream_t stream);

// FP32 logits [n][v_t] -> loss [n], and the rows overwritten in place with the
// softmax over the whole vocabulary (LSE combined with peer_lse when given).
hipError_t xent_probs(float* logits, int64_t n, int32_t v_t, int64_t v0, const int64_t* targets,
                      const float* peer_lse, const float* peer_z, float* loss, hipStream_t stream);
// dlogits (bf16 [n][v_t]) = (softmax - onehot(target)) * grad_scale.
hipError_t xent_grad(const float* probs, int64_t n, int32_t v_t, int64_t v0, const int64_t* targets,
                     float grad_scale, uint16_t* dlogits, hipStream_t stream);

// ---------------------------------------------------------------- embedding

// Gathered row m (0 <= m < rows = b*s_c) of the vocabulary-parallel lookup:
// w[ids[m] - v0] if in [0, v_t) else 0; own SP rows -> own (+ receipt), the
// peers' rows -> send (row mapping as RowSrc).
hipError_t embed_fwd(const int64_t* ids, const uint16_t* w, int64_t v0, int32_t v_t, int32_t h, int64_t rows,
                     int32_t s_c, int32_t s_sp, int32_t r, int32_t t, const uint16_t* receipt, uint16_t* own,
                     uint16_t* send, hipStream_t stream);
// Rows of an fp32 [rows][h] sum over the gathered view: own SP rows ->
// bf16(sum + receipt) into own (receipt may be null), the peers' rows ->
// bf16(sum) into send (row mapping as RowSrc).
hipError_t sp_finish(const float* sum, int32_t h, int64_t rows, int32_t s_c, int32_t s_sp, int32_t r, int32_t t,
                     const uint16_t* receipt, uint16_t* own, uint16_t* send, hipStream_t stream);
// dw[ids[m] - v0] += dy.row(m) for the ids in range (fp32 atomics).
hipError_t embed_bwd(const int64_t* ids, RowSrc dy, int64_t v0, int32_t v_t, int32_t h, int64_t rows, float* dw,
                     hipStream_t stream);

// ---------------------------------------------------------------- optimizer

// Step constants of one Adam step, prepared on the host in double precision.
struct AdamConsts {
  float beta1, beta2, one_m_beta1, one_m_beta2;
  float lr, decay;           // decay = lr * weight_decay
  float r1, rs2;             // 1 / (1 - beta1^t), 1 / sqrt(1 - beta2^t)
  float eps, scale;
  const float* scale_dev;    // device scalar multiplying scale, or null
};
// grad, master, m, v: f32 [n], 16-byte aligned; weight: bf16 [n], 8-byte aligned.
hipError_t adam_step(const AdamConsts& c, int64_t n, float* grad, float* master, float* m, float* v,
                     uint16_t* weight, int32_t zero_grad, hipStream_t stream);

}  // namespace l4d
