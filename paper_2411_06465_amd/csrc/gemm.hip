// bf16 GEMM on the gfx950 matrix cores: C[m][n] = sum_k A(m,k) B(n,k), fp32
// accumulation, with the layer's fused epilogues.
//
// A workgroup owns a 256x256 tile of C; each wave accumulates a 128 x (NS*32)
// block as tiles of v_mfma_f32_32x32x16_bf16.  Operand tiles move global ->
// LDS by global_load_lds_dwordx4 (direct-to-LDS DMA, one contiguous KB per
// wave instruction, no staging registers).  Every stage buffer is its own LDS
// object, so the compiler knows a read of one stage cannot depend on the
// copies still landing in the others.  Two kernels:
//
//  * gemm_bk64 (K a multiple of 128): two stages of 64 k.  A K-contiguous copy
//    moves 8 whole 128-byte rows per instruction (one cache line each); the
//    fragments of the next 16-k sub-step are read from LDS under the MFMAs of
//    the current one, and the barrier that publishes stage kt+1 sits before
//    the last sub-step of stage kt, right after which the freed buffers take
//    stage kt+2 (the A half there, the B half one sub-step later, so the
//    copies do not all reach the texture path at once).  8 waves (two per
//    SIMD, 128x64 each) or 4 (128x128 each).
//  * gemm_bk32 (any K that is a multiple of 8): 8 waves, four stages of 32 k,
//    16 rows x 64 bytes per copy instruction, the stage past K zeroed in
//    registers.
//
// Operand layouts: "KC" (reduction index contiguous: activations in the
// forward, the output gradient in dX) is stored row by row, the 16-byte chunks
// of a row permuted by an XOR with row bits so that the 16 rows a 16-lane
// group of a fragment read touches cover all 64 banks (256 bytes) once.  "MN" (reduction
// index strided: the weight in dX, both operands of dW) is stored as k-rows
// of 256 columns with the 16-byte chunks XOR-swizzled by row, and read with
// two ds_read_b64_tr_b16 that hand each lane 4 consecutive k of one column --
// the transpose happens in the LDS read, not in registers.
//
// A wave's 32-column blocks come in pairs PAIR columns apart, so the columns
// n and n + PAIR land in the same lane and register: a RoPE pair (i, i + d_h/2)
// or a gate/up pair of the fused FFN weight.  The epilogue stages rows through
// LDS and hands 8-column vectors to the fused operation, with that operation's
// global inputs loaded for a whole pass first.  The fp32 accumulate (dW) needs
// no staging: the C tile meets the accumulators in registers (added at the end
// in the BK = 64 kernel, loaded before the first product in the BK = 32 one).
#include "kernels.h"

namespace l4d {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define GPTR(p) ((const __attribute__((address_space(1))) void*)(p))
#define LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int TILE_BYTES = 256 * BK * 2;     // 16 KB per operand per stage
constexpr int GROUP_M = 4;

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Direct-to-LDS copy: 16 bytes per lane from g into the wave's 1 KB LDS chunk
// at lds (lane i lands at byte 16 i).  Inline assembly, so that the compiler's
// wait-count pass does not see an LDS write in flight: it cannot tell one
// stage buffer from another and would wait for every copy before the first
// LDS read of the next stage, exposing the copy latency on every stage.  The
// kernels wait for their own copies (vmcnt) before the barrier that publishes
// a stage, and before the stages are reused as epilogue staging space.
// TAG only changes the asm text (a comment), to keep copies in the two arms of
// a branch from being merged.
template <int TAG = 0>
__device__ __forceinline__ void dma16(const uint16_t* g, const uint8_t* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(   // uniform by construction; stated for the compiler
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(LPTR(const_cast<uint8_t*>(lds)))));
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off ; copy form %2" ::"v"(g), "s"(l), "n"(TAG)
               : "memory", "m0");
}

__device__ __forceinline__ u32x4 pack8(const float* v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{v[2 * i], v[2 * i + 1]}, bf16x2));
  return r;
}
__device__ __forceinline__ void unpack8(u32x4 u, float* v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(u[i] << 16);
    v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
  const int X = 8;   // workgroups go round-robin over the 8 XCDs; give each a contiguous tile range
  int per = nwg / X, rem = nwg % X, xcd = bid % X, local = bid / X;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// ------------------------------------------------------------------ LDS layouts
// KC tile: row r (0..255) holds its 32 k (64 bytes) at r*64, the four 16-byte
// chunks permuted by c ^ ((r >> 2) & 3).  Four rows share a 256-byte bank line
// (r % 4 picks the quarter), so the 16 rows one 16-lane group of a fragment
// read touches cover all 64 banks once.
__device__ __forceinline__ int kc_off(int row, int chunk) { return row * 64 + ((chunk ^ ((row >> 2) & 3)) << 4); }
// MN tile: k-row r (0..31), 16-byte chunk c (0..31) of its 256 columns,
// stored at chunk c ^ 4 (r % 4).  A transposing read (32 lanes: 4 k-rows x an
// aligned group of 4 chunks) then touches 4 different chunk groups, all 64
// banks once; k-rows r and r + 4 share the pattern.
__device__ __forceinline__ int mn_swz(int row) { return (row & 3) << 2; }
__device__ __forceinline__ int mn_off(int row, int chunk) { return row * 512 + ((chunk ^ mn_swz(row)) << 4); }

// Each stage holds 16 KB per operand; wave w copies LDS KB numbers
// kb = w + WAVES * q.  KC: KB kb holds tile rows 16 kb + lane/4, 64 contiguous
// bytes of each row per instruction (4 lanes), lane l fetching the chunk
// that belongs at its LDS slot l % 4: chunk (l & 3) ^ ((l >> 4) & 3), the
// same for every q.  A lane's source rows are fixed over K and kept as
// pointers.  MN: KB kb holds k-rows 2 kb + lane/32.
template <int WAVES>
struct KcRows {
  const uint16_t* row[16 / WAVES];   // source row of copy q (chunk not included)
  int c8;                            // element offset of the lane's chunk
};

template <int WAVES>
__device__ __forceinline__ KcRows<WAVES> kc_rows(const Operand& op, int x0, int tile_idx, int wave, int lane) {
  KcRows<WAVES> r;
  r.c8 = 8 * ((lane & 3) ^ ((lane >> 4) & 3));
#pragma unroll
  for (int q = 0; q < 16 / WAVES; ++q) {
    const int xr = 16 * (wave + WAVES * q) + (lane >> 2);
    int64_t gx;
    if (op.split_rows) {
      int i = tile_idx * 128 + (xr & 127);
      if (i >= op.split_rows) i = op.split_rows - 1;
      gx = (xr >= 128 ? op.split_off : 0) + i;
    } else {
      gx = x0 + xr;
      if (gx >= op.rows) gx = op.rows - 1;
    }
    r.row[q] = op.src.row(gx);
  }
  return r;
}

// RAGGED: K may end inside the stage; the chunks past K copy the last whole
// chunk instead (those fragments are zeroed before use).
template <int WAVES, bool RAGGED>
__device__ __forceinline__ void copy_kc(uint8_t* lds, const KcRows<WAVES>& rows, int k0, int K, int wave) {
  int k = k0 + rows.c8;
  if constexpr (RAGGED) k = min(k, K - 8);
#pragma unroll
  for (int q = 0; q < 16 / WAVES; ++q)
    dma16(rows.row[q] + k, lds + (wave + WAVES * q) * 1024);
}

template <int WAVES>
__device__ __forceinline__ void copy_mn(uint8_t* lds, const Operand& op, int x0, int k0, int K, int wave,
                                        int lane) {
#pragma unroll
  for (int q = 0; q < 16 / WAVES; ++q) {
    const int kb = wave + WAVES * q;
    const int kr = 2 * kb + (lane >> 5);
    const int lc = (lane & 31) ^ mn_swz(kr);
    int k = k0 + kr;
    if (k >= K) k = K - 1;
    int x = x0 + lc * 8;
    if (x >= op.rows) x = op.rows - 8;
    const uint32_t o = op.src.row_index(k);
    const uint16_t* base = (o & 0x80000000u) ? op.src.peer : op.src.own;
    dma16(base + static_cast<int64_t>(o & 0x7fffffffu) * op.src.ld + x, lds + kb * 1024);
  }
}

// MFMA operand for rows x0 + lane%32 (x0 a multiple of 32), k = 16 kk + 8 (lane/32) + 0..7.
template <Layout L>
__device__ __forceinline__ bf16x8 frag(const uint8_t* lds, int x0, int kk, int lane) {
  if constexpr (L == Layout::KC) {
    return *reinterpret_cast<const bf16x8*>(lds + kc_off(x0 + (lane & 31), 2 * kk + (lane >> 5)));
  } else {
    const int li = lane & 15;
    const int row = 16 * kk + 8 * (lane >> 5) + (li >> 2);
    const int x = x0 + 16 * ((lane >> 4) & 1) + 4 * (li & 3);
    const int off = mn_off(row, x >> 3) + ((x & 7) << 1);
    const int off4 = mn_off(row + 4, x >> 3) + ((x & 7) << 1);
    const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) i16x4*>(LPTR(const_cast<uint8_t*>(lds) + off)));
    const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        reinterpret_cast<__attribute__((address_space(3))) i16x4*>(LPTR(const_cast<uint8_t*>(lds) + off4)));
    const u32x2 ua = __builtin_bit_cast(u32x2, a), ub = __builtin_bit_cast(u32x2, b);
    return __builtin_bit_cast(bf16x8, u32x4{ua[0], ua[1], ub[0], ub[1]});
  }
}

// -------------------------------------------------------------- epilogues

// silu(g) = g * sigmoid(g); the reciprocal is the hardware one (1 ulp), far
// below the bf16 rounding of every value it feeds.
__device__ __forceinline__ float sigmoid_f(float g) { return __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// Global inputs of one epilogue call (8 columns at `col` and the 8 PAIR
// further), loaded for a whole pass of the staged epilogue before the tile is
// staged, so that their latencies overlap instead of adding up.
template <EpiKind KIND>
struct EpiIn {};
template <>
struct EpiIn<EpiKind::ResidualSP> {
  u32x4 r[2], q[2];       // residual, receipt: low and high half
};
template <>
struct EpiIn<EpiKind::SwiGLUBwd> {
  u32x4 g[2], u[2], a[2];
};
template <>
struct EpiIn<EpiKind::QkvRope> {
  float4 cs[4];           // (cos, sin) of the 8 columns
};

// Output row of logical row m for ResidualSP: own rows map into own_out,
// the others into the send buffer.
__device__ __forceinline__ int64_t resid_row(const EpiParams& e, int64_t m, bool& own) {
  own = true;
  if (e.t == 1) return m;
  const int64_t bi = m / e.s_c;
  const int32_t i = static_cast<int32_t>(m - bi * e.s_c);
  const int32_t lo_row = e.r * e.s_sp;
  own = i >= lo_row && i < lo_row + e.s_sp;
  return own ? bi * e.s_sp + (i - lo_row) : bi * static_cast<int64_t>(e.t - 1) * e.s_sp + (i < lo_row ? i : i - e.s_sp);
}

template <EpiKind KIND, int PAIR>
__device__ __forceinline__ void epi_load(const GemmParams& p, int64_t m, int tn, int col, EpiIn<KIND>& in) {
  const EpiParams& e = p.epi;
  if (m >= p.M) return;
  const int n_lo = tn * BN + col;
  if constexpr (KIND == EpiKind::ResidualSP) {
    bool own;
    const int64_t orow = resid_row(e, m, own);
    if (!own) return;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = n_lo + h * PAIR;
      if (n >= p.N) continue;
      const int64_t off = orow * e.ldc + n;
      if (e.resid) in.r[h] = *reinterpret_cast<const u32x4*>(e.resid + off);
      if (e.receipt) in.q[h] = *reinterpret_cast<const u32x4*>(e.receipt + off);
    }
  } else if constexpr (KIND == EpiKind::SwiGLUBwd) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = n_lo + h * PAIR;
      if (n >= p.N) continue;
      const int64_t off = m * e.f + n;
      in.g[h] = *reinterpret_cast<const u32x4*>(e.g_in + off);
      in.u[h] = *reinterpret_cast<const u32x4*>(e.u_in + off);
      in.a[h] = *reinterpret_cast<const u32x4*>(e.act_in + off);
    }
  } else if constexpr (KIND == EpiKind::QkvRope) {
    if (n_lo >= p.N || n_lo >= e.nq + e.nk) return;     // V columns are not rotated
    const int n = n_lo < e.nq ? n_lo : n_lo - e.nq;
    const int32_t i = static_cast<int32_t>(m % e.s_c);
    const float4* tab = reinterpret_cast<const float4*>(e.rope + static_cast<int64_t>(i) * (e.d_h / 2) + (n % e.d_h));
#pragma unroll
    for (int j = 0; j < 4; ++j) in.cs[j] = tab[j];
  }
}

// lo: 8 columns starting at tile column `col`; hi: the 8 columns PAIR further.
template <EpiKind KIND, int PAIR>
__device__ __forceinline__ void epilogue(const GemmParams& p, int64_t m, int tn, int col, float* lo, float* hi,
                                         const EpiIn<KIND>& in) {
  const EpiParams& e = p.epi;
  if (m >= p.M) return;
  const int n_lo = tn * BN + col;
  switch (KIND) {
    case EpiKind::StoreBF16: {
      uint16_t* c = static_cast<uint16_t*>(e.c) + m * e.ldc;
      if (n_lo < p.N) *reinterpret_cast<u32x4*>(c + n_lo) = pack8(lo);
      if (n_lo + PAIR < p.N) *reinterpret_cast<u32x4*>(c + n_lo + PAIR) = pack8(hi);
      break;
    }
    case EpiKind::StoreF32: {
      float* c = static_cast<float*>(e.c) + m * e.ldc;
      if (n_lo < p.N) {
        *reinterpret_cast<float4*>(c + n_lo) = make_float4(lo[0], lo[1], lo[2], lo[3]);
        *reinterpret_cast<float4*>(c + n_lo + 4) = make_float4(lo[4], lo[5], lo[6], lo[7]);
      }
      if (n_lo + PAIR < p.N) {
        *reinterpret_cast<float4*>(c + n_lo + PAIR) = make_float4(hi[0], hi[1], hi[2], hi[3]);
        *reinterpret_cast<float4*>(c + n_lo + PAIR + 4) = make_float4(hi[4], hi[5], hi[6], hi[7]);
      }
      break;
    }
    case EpiKind::AccF32:     // handled in registers (acc_load_f32 / acc_store_f32)
      break;
    case EpiKind::QkvRope: {
      if constexpr (KIND == EpiKind::QkvRope) {
        // n_lo lies in the first half of a head, n_lo + PAIR (PAIR = d_h/2) in the second.
        if (n_lo >= p.N) break;
        uint16_t* dst;
        int64_t ld;
        int n;
        bool rot = true;
        if (n_lo < e.nq) { dst = e.q; ld = e.nq; n = n_lo; }
        else if (n_lo < e.nq + e.nk) { dst = e.k; ld = e.nk; n = n_lo - e.nq; }
        else { dst = e.v; ld = e.nk; n = n_lo - e.nq - e.nk; rot = false; }
        if (rot) {
          float a[8], b[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float c = j & 1 ? in.cs[j >> 1].z : in.cs[j >> 1].x;
            const float sn = j & 1 ? in.cs[j >> 1].w : in.cs[j >> 1].y;
            a[j] = lo[j] * c - hi[j] * sn;
            b[j] = hi[j] * c + lo[j] * sn;
          }
          *reinterpret_cast<u32x4*>(dst + m * ld + n) = pack8(a);
          *reinterpret_cast<u32x4*>(dst + m * ld + n + PAIR) = pack8(b);
        } else {
          *reinterpret_cast<u32x4*>(dst + m * ld + n) = pack8(lo);
          *reinterpret_cast<u32x4*>(dst + m * ld + n + PAIR) = pack8(hi);
        }
      }
      break;
    }
    case EpiKind::ResidualSP: {
      if constexpr (KIND == EpiKind::ResidualSP) {
        bool own;
        const int64_t orow = resid_row(e, m, own);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int n = n_lo + h * PAIR;
          if (n >= p.N) continue;
          float* src = h ? hi : lo;
          const int64_t off = orow * e.ldc + n;
          if (own) {
            float r[8];
            if (e.resid) {
              unpack8(in.r[h], r);
#pragma unroll
              for (int j = 0; j < 8; ++j) src[j] += r[j];
            }
            if (e.receipt) {
              unpack8(in.q[h], r);
#pragma unroll
              for (int j = 0; j < 8; ++j) src[j] += r[j];
            }
            if (e.own_out_f32) {
              float4* o32 = reinterpret_cast<float4*>(e.own_out_f32 + off);
              o32[0] = make_float4(src[0], src[1], src[2], src[3]);
              o32[1] = make_float4(src[4], src[5], src[6], src[7]);
            } else {
              *reinterpret_cast<u32x4*>(e.own_out + off) = pack8(src);
            }
          } else {
            *reinterpret_cast<u32x4*>(e.send + off) = pack8(src);
          }
        }
      }
      break;
    }
    case EpiKind::SwiGLUFwd: {
      const int j = tn * 128 + col;       // FFN column of this gate/up pair
      if (j >= e.f) break;
      const int64_t off = m * e.f + j;
      float g[8], u[8], a[8], pr[8];
      unpack8(pack8(lo), g);              // the stored (rounded) G and U feed act and prod
      unpack8(pack8(hi), u);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        a[q] = g[q] * sigmoid_f(g[q]);
        pr[q] = a[q] * u[q];
      }
      *reinterpret_cast<u32x4*>(e.g_out + off) = pack8(g);
      *reinterpret_cast<u32x4*>(e.u_out + off) = pack8(u);
      *reinterpret_cast<u32x4*>(e.act_out + off) = pack8(a);
      *reinterpret_cast<u32x4*>(e.prod_out + off) = pack8(pr);
      break;
    }
    case EpiKind::SwiGLUBwd: {
      if constexpr (KIND == EpiKind::SwiGLUBwd) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int n = n_lo + h * PAIR;
          if (n >= p.N) continue;
          const float* dp = h ? hi : lo;
          const int64_t off = m * e.f + n;
          float g[8], u[8], a[8], dg[8], du[8];
          unpack8(in.g[h], g);
          unpack8(in.u[h], u);
          unpack8(in.a[h], a);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float s = sigmoid_f(g[q]);
            dg[q] = dp[q] * u[q] * (s * (1.0f + g[q] * (1.0f - s)));
            du[q] = dp[q] * a[q];
          }
          uint16_t* out = e.dgu + m * (2 * static_cast<int64_t>(e.f));
          *reinterpret_cast<u32x4*>(out + n) = pack8(dg);
          *reinterpret_cast<u32x4*>(out + e.f + n) = pack8(du);
        }
      }
      break;
    }
  }
}

// Tile column of a wave's low 32-column block j; its partner is PAIR further.
// 8 waves: wn = 0..3, one low block each; 4 waves: wn = 0..1, two each.
template <int WAVES, int PAIR>
__device__ __forceinline__ int lo_col(int wn, int j) {
  if constexpr (WAVES == 8) {
    constexpr int PW = PAIR / 32;
    return (wn / PW) * (2 * PAIR) + (wn % PW) * 32;
  } else {
    if constexpr (PAIR == 32) return wn * 128 + j * 64;
    else if constexpr (PAIR == 64) return wn * 128 + j * 32;
    else return wn * 64 + j * 32;
  }
}

// -------------------------------------------------------------- the kernels

// Workgroup barrier between pipeline steps.  __syncthreads() would also fence
// global memory, i.e. wait for every copy still in flight -- including the
// stages being prefetched; each wave has already waited for its own copies of
// the step that is about to be read, so only the LDS reads of the previous
// step (lgkmcnt) must drain before the barrier.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 4) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
}

// Epilogue: each wave stages R rows x (NS*32) columns of fp32 at a time in its
// own 16 KB of LDS (column halves swapped on rows with bit 2 set, so the two
// half-waves write different banks) and hands out 8-column vectors of its low
// blocks with their PAIR partners.  Accumulator register i of a lane: row
// 8(i/4) + 4(lane/32) + i%4, column lane%32 of its 32x32 tile.  The global
// inputs of a pass are loaded before its rows are staged.
template <EpiKind KIND, int PAIR, int NS>
__device__ __forceinline__ void store_tile(const GemmParams& p, f32x16 (&acc)[4][NS], float* st, int64_t row0,
                                           int tn, const int* ncol, int lane) {
  constexpr int C = NS * 32, R = 4096 / C, PASSES = 128 / R, MS_PER = R / 32;
  constexpr int VEC = R * (NS / 2) * 4;  // 8-column vectors of the low blocks per pass
  constexpr int ITERS = VEC / 64;
#pragma unroll
  for (int pass = 0; pass < PASSES; ++pass) {
    EpiIn<KIND> in[ITERS];
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int idx = it * 64 + lane;
      const int rr = idx / ((NS / 2) * 4), v = idx % ((NS / 2) * 4);
      epi_load<KIND, PAIR>(p, row0 + pass * R + rr, tn, ncol[v >> 2] + (v & 3) * 8, in[it]);
    }
#pragma unroll
    for (int mm = 0; mm < MS_PER; ++mm)
#pragma unroll
      for (int ns = 0; ns < NS; ++ns)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = mm * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
          const int cc = (ns * 32 + (lane & 31)) ^ (((r >> 2) & 1) << 4);
          st[r * C + cc] = acc[pass * MS_PER + mm][ns][i];
        }
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int idx = it * 64 + lane;
      const int rr = idx / ((NS / 2) * 4), v = idx % ((NS / 2) * 4);
      const int j = v >> 2, c8 = (v & 3) * 8;
      const int flip = ((rr >> 2) & 1) << 4;
      const float4* lo4 = reinterpret_cast<const float4*>(st + rr * C + ((j * 32 + c8) ^ flip));
      const float4* hi4 = reinterpret_cast<const float4*>(st + rr * C + (((j + NS / 2) * 32 + c8) ^ flip));
      const float4 l0 = lo4[0], l1 = lo4[1], h0 = hi4[0], h1 = hi4[1];
      float lo[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
      float hi[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
      epilogue<KIND, PAIR>(p, row0 + pass * R + rr, tn, ncol[j] + c8, lo, hi, in[it]);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
  }
}

// AccF32 (C += A B^T in fp32) works on the accumulators directly.  In the BK =
// 32 kernel the tile of C is loaded into them before the first product (its
// latency overlaps the first stage's copies) and stored from them at the end;
// the BK = 64 kernel adds it at the end (acc_add_store_f32).  In the accumulator layout
// the 32 lanes of a half-wave cover 32 consecutive columns (128 bytes) of one
// row, so both are whole-line accesses without staging.  Whole tiles load and
// store non-temporally: each C element is touched once per launch, and
// streaming it leaves L2 to the operand tiles the neighbouring workgroups share
// (4-5% off the largest weight-gradient GEMM of the Llama-2-7B layer).
template <int NS>
__device__ __forceinline__ void acc_load_f32(f32x16 (&acc)[4][NS], const GemmParams& p, const float* cbase,
                                             int64_t ldc, int64_t row0, int tn, const int* ncol, int lane) {
  const int rl = 4 * (lane >> 5);
  int32_t off[NS];            // lane's element offset from its row block's first row
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) off[ns] = static_cast<int32_t>(rl * ldc) + tn * BN + ncol[ns] + (lane & 31);
  const bool full = row0 + 128 <= p.M && (tn + 1) * BN <= p.N;   // uniform
  if (full) {
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = ms * 32 + 8 * (i >> 2) + (i & 3);
        const float* row = cbase + (row0 + r) * ldc;   // uniform
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) acc[ms][ns][i] = __builtin_nontemporal_load(&row[off[ns]]);
      }
  } else {
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = ms * 32 + 8 * (i >> 2) + (i & 3);
        const float* row = cbase + (row0 + r) * ldc;   // uniform
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) {
          const int n = tn * BN + ncol[ns] + (lane & 31);
          acc[ms][ns][i] = (row0 + r + rl < p.M && n < p.N) ? row[off[ns]] : 0.0f;
        }
      }
  }
}

template <int NS>
__device__ __forceinline__ void acc_store_f32(const f32x16 (&acc)[4][NS], const GemmParams& p, float* cbase,
                                              int64_t ldc, int64_t row0, int tn, const int* ncol, int lane) {
  const int rl = 4 * (lane >> 5);
  int32_t off[NS];
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) off[ns] = static_cast<int32_t>(rl * ldc) + tn * BN + ncol[ns] + (lane & 31);
  const bool full = row0 + 128 <= p.M && (tn + 1) * BN <= p.N;
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = ms * 32 + 8 * (i >> 2) + (i & 3);
      float* row = cbase + (row0 + r) * ldc;
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) {
        const int n = tn * BN + ncol[ns] + (lane & 31);
        if (full || (row0 + r + rl < p.M && n < p.N)) __builtin_nontemporal_store(acc[ms][ns][i], &row[off[ns]]);
      }
    }
}

// acc + C -> C for a tile whose products started from zero, one accumulator
// row block (32 rows) at a time.  Whole tiles are software-pipelined: the
// loads of block ms + 1 are issued before the stores of block ms, so that
// waiting for a block's C values (the wait counter also counts stores) does
// not wait for the stores issued after them.  They go through a buffer
// descriptor of the wave's 128 rows: the row offset is a scalar, the lane
// offset one register per column block, which leaves the registers for the
// two blocks of C in flight.  Edge tiles go element by element.
constexpr int kBufNT = 2;   // cache-policy bit of a non-temporal buffer access
template <int NS>
__device__ __forceinline__ void acc_add_store_f32(const f32x16 (&acc)[4][NS], const GemmParams& p, float* cbase,
                                                  int64_t ldc, int64_t row0, int tn, const int* ncol, int lane) {
  const int rl = 4 * (lane >> 5);
  if (row0 + 128 <= p.M && (tn + 1) * BN <= p.N) {   // uniform
    const __amdgpu_buffer_rsrc_t win =
        __builtin_amdgcn_make_buffer_rsrc(cbase + row0 * ldc, 0, static_cast<int>(0x7fffffff), 0x00020000);
    int32_t voff[NS];   // lane's byte offset in its row
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) voff[ns] = (static_cast<int32_t>(rl * ldc) + tn * BN + ncol[ns] + (lane & 31)) * 4;
    const int32_t ldc4 = static_cast<int32_t>(ldc * 4);
    float c[2][16][NS];   // the buffer builtins move 32-bit words: bit casts, not conversions
    auto load = [&](int ms, float (&cb)[16][NS]) {
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int ns = 0; ns < NS; ++ns)
          cb[i][ns] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                       win, voff[ns], (ms * 32 + 8 * (i >> 2) + (i & 3)) * ldc4, kBufNT));
    };
    load(0, c[0]);
#pragma unroll
    for (int ms = 0; ms < 4; ++ms) {
      if (ms + 1 < 4) load(ms + 1, c[(ms + 1) & 1]);
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int ns = 0; ns < NS; ++ns)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, acc[ms][ns][i] + c[ms & 1][i][ns]), win,
                                                voff[ns], (ms * 32 + 8 * (i >> 2) + (i & 3)) * ldc4, kBufNT);
    }
    return;
  }
  int32_t off[NS];
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) off[ns] = static_cast<int32_t>(rl * ldc) + tn * BN + ncol[ns] + (lane & 31);
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = ms * 32 + 8 * (i >> 2) + (i & 3);
      float* row = cbase + (row0 + r) * ldc;
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) {
        const int n = tn * BN + ncol[ns] + (lane & 31);
        if (row0 + r + rl < p.M && n < p.N) row[off[ns]] += acc[ms][ns][i];
      }
    }
}

// Ends the accumulators' pending loads here: an asm that reads and redefines
// them makes the compiler wait for the loads before it, once, instead of at
// their first use inside the main loop on every iteration (where the counter
// also holds the copies of the next stages).
template <int NS>
__device__ __forceinline__ void settle_acc(f32x16 (&acc)[4][NS]) {
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) asm volatile("" : "+v"(acc[ms][ns]));
}

struct TileCoord {
  int tm, tn;
};
// Tile `pid` in the grouped order: GROUP_M tile rows at a time, column by column.
__device__ __forceinline__ TileCoord tile_coord(const GemmParams& p, int pid) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.B.split_rows ? (p.B.split_rows + 127) / 128 : (p.N + BN - 1) / BN;
  const int group = GROUP_M * tiles_n;
  const int first_m = (pid / group) * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  return TileCoord{first_m + (pid % group) % gm, (pid % group) / gm};
}
__device__ __forceinline__ TileCoord tile_of(const GemmParams& p) {
  return tile_coord(p, xcd_remap(blockIdx.x, gridDim.x));
}

// 8 waves (two per SIMD), each 128 x 64.
template <Layout LA, Layout LB, EpiKind KIND, int PAIR>
__global__ void __launch_bounds__(512, 1) gemm_bk32(GemmParams p) {
  constexpr int WAVES = 8, NS = 2, PER = 2;
  constexpr bool RAGGED = true;
  __shared__ __attribute__((aligned(16))) uint8_t a0[TILE_BYTES], b0[TILE_BYTES], a1[TILE_BYTES], b1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t a2[TILE_BYTES], b2[TILE_BYTES], a3[TILE_BYTES], b3[TILE_BYTES];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave: scalar code for wave-level decisions
  const TileCoord tc = tile_of(p);
  const int tm = tc.tm, tn = tc.tn, m0 = tm * BM, n0 = tn * BN;
  const int wm = wave >> 2, wn = wave & 3;
  int ncol[NS];
  ncol[0] = lo_col<WAVES, PAIR>(wn, 0);
  ncol[1] = ncol[0] + PAIR;

  f32x16 acc[4][NS];
  if constexpr (KIND == EpiKind::AccF32) {
    acc_load_f32<NS>(acc, p, static_cast<float*>(p.epi.c), p.epi.ldc, static_cast<int64_t>(m0) + wm * 128, tn,
                     ncol, lane);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NS; ++j) acc[i][j] = f32x16{};
  }

  KcRows<WAVES> ra{}, rb{};
  if constexpr (LA == Layout::KC) ra = kc_rows<WAVES>(p.A, m0, tm, wave, lane);
  if constexpr (LB == Layout::KC) rb = kc_rows<WAVES>(p.B, n0, tn, wave, lane);

  auto issue = [&](int k0, uint8_t* la, uint8_t* lb) {
    if constexpr (LA == Layout::KC) copy_kc<WAVES, RAGGED>(la, ra, k0, p.K, wave);
    else copy_mn<WAVES>(la, p.A, m0, k0, p.K, wave, lane);
    if constexpr (LB == Layout::KC) copy_kc<WAVES, RAGGED>(lb, rb, k0, p.K, wave);
    else copy_mn<WAVES>(lb, p.B, n0, k0, p.K, wave, lane);
  };
  auto compute = [&](int k0, const uint8_t* la, const uint8_t* lb) {
    const bool tail = k0 + BK > p.K;     // uniform: only the last step of a ragged K
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[4], bf[NS];
#pragma unroll
      for (int ms = 0; ms < 4; ++ms) af[ms] = frag<LA>(la, wm * 128 + ms * 32, kk, lane);
#pragma unroll
      for (int ns = 0; ns < NS; ++ns) bf[ns] = frag<LB>(lb, ncol[ns], kk, lane);
      if (tail) {
        const bool z = k0 + 16 * kk + 8 * (lane >> 5) >= p.K;
#pragma unroll
        for (int ms = 0; ms < 4; ++ms) af[ms] = z ? bf16x8{} : af[ms];
#pragma unroll
        for (int ns = 0; ns < NS; ++ns) bf[ns] = z ? bf16x8{} : bf[ns];
      }
#pragma unroll
      for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int ns = 0; ns < NS; ++ns)
          acc[ms][ns] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ms], bf[ns], acc[ms][ns], 0, 0, 0);
    }
  };

  // Step kt reads stage kt % 4.  On entry to a step the copies of the next two
  // steps may still be in flight (2 * PER instructions per operand each):
  // wait until only those remain, then a barrier makes every wave's copy of
  // this step visible and frees the stage of step kt - 1 for step kt + 3.
  const int nk = (p.K + BK - 1) / BK;
  auto step = [&](int kt, const uint8_t* la, const uint8_t* lb, uint8_t* na, uint8_t* nb) {
    const int after = nk - 1 - kt;
    if (after >= 2) wait_vm<4 * PER>();
    else if (after == 1) wait_vm<2 * PER>();
    else wait_vm<0>();
    stage_barrier();
    if (kt + 3 < nk) issue((kt + 3) * BK, na, nb);
    __builtin_amdgcn_sched_barrier(0);   // the copies go out now, not next to the wait for them
    compute(kt * BK, la, lb);
  };
  issue(0, a0, b0);
  if constexpr (KIND == EpiKind::AccF32) settle_acc<NS>(acc);   // the C tile (and stage 0) have landed
  if (nk > 1) issue(BK, a1, b1);
  if (nk > 2) issue(2 * BK, a2, b2);
  // Whole groups of 4 steps without early exits (an exit between the unrolled
  // steps makes the register allocator spill), then the remaining 0-3 steps.
  int kt = 0;
  for (; kt + 4 <= nk; kt += 4) {
    step(kt, a0, b0, a3, b3);
    step(kt + 1, a1, b1, a0, b0);
    step(kt + 2, a2, b2, a1, b1);
    step(kt + 3, a3, b3, a2, b2);
  }
  const int rest = nk - kt;
  if (rest > 0) step(kt, a0, b0, a3, b3);
  if (rest > 1) step(kt + 1, a1, b1, a0, b0);
  if (rest > 2) step(kt + 2, a2, b2, a1, b1);
  wait_vm<0>();      // no copy may land in the stages once they are staging space (or after the end)
  if constexpr (KIND == EpiKind::AccF32) {
    acc_store_f32<NS>(acc, p, static_cast<float*>(p.epi.c), p.epi.ldc, static_cast<int64_t>(m0) + wm * 128, tn,
                      ncol, lane);
  } else {
    __syncthreads();   // every wave is done reading the stages before they become staging space
    uint8_t* mine = wave == 0 ? a0 : wave == 1 ? b0 : wave == 2 ? a1 : wave == 3 ? b1 : wave == 4 ? a2
                  : wave == 5 ? b2 : wave == 6 ? a3 : b3;
    store_tile<KIND, PAIR, NS>(p, acc, reinterpret_cast<float*>(mine), static_cast<int64_t>(m0) + wm * 128, tn,
                               ncol, lane);
  }
}

// ---------------------------------------------------------- BK = 64 variant
// Two stages of 64 k (32 KB per operand each, 128 KB in all).  A KC copy
// instruction moves 8 whole rows of 128 bytes (one cache line each, so no
// line is fetched twice); an MN copy instruction moves 2 k-rows of 512 bytes.
// KC slot s of row r holds chunk s ^ ((r >> 1) & 7).  Two rows share a 256-byte
// bank line (r % 2 picks the half), so the 16 rows one 16-lane group of a
// fragment read touches cover all 64 banks once.
constexpr int BK2 = 64;
constexpr int TILE2 = 256 * BK2 * 2;     // 32 KB per operand per stage

__device__ __forceinline__ int kc2_off(int row, int chunk) { return row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4); }

template <int WAVES>
struct Kc2Rows {
  const uint16_t* row[32 / WAVES];
  int c8;
};

// Copy q of wave w moves rows 8 kb + lane/8, kb = w + WAVES q; (row >> 1) & 7 =
// 4 (w & 1) + lane/16 is the same for every q.
template <int WAVES>
__device__ __forceinline__ Kc2Rows<WAVES> kc2_rows(const Operand& op, int x0, int tile_idx, int wave, int lane) {
  Kc2Rows<WAVES> r;
  r.c8 = 8 * ((lane & 7) ^ (4 * (wave & 1) + (lane >> 4)));
#pragma unroll
  for (int q = 0; q < 32 / WAVES; ++q) {
    const int xr = 8 * (wave + WAVES * q) + (lane >> 3);
    int64_t gx;
    if (op.split_rows) {
      int i = tile_idx * 128 + (xr & 127);
      if (i >= op.split_rows) i = op.split_rows - 1;
      gx = (xr >= 128 ? op.split_off : 0) + i;
    } else {
      gx = x0 + xr;
      if (gx >= op.rows) gx = op.rows - 1;
    }
    r.row[q] = op.src.row(gx);
  }
  return r;
}

template <int WAVES>
__device__ __forceinline__ void copy2_kc(uint8_t* lds, const Kc2Rows<WAVES>& rows, int k0, int wave) {
  const int k = k0 + rows.c8;
#pragma unroll
  for (int q = 0; q < 32 / WAVES; ++q)
    dma16(rows.row[q] + k, lds + (wave + WAVES * q) * 1024);
}

// MN copies.  For an operand whose rows are one plain array (no sequence-
// parallel split) a lane's offset is fixed over K and across its copies up to
// a uniform stride: copy q reads k-row kr0 + 2 * WAVES * q, and the column
// swizzle depends on kr mod 4, which q does not change.  One offset per lane
// is kept; each stage adds one uniform row offset.  A split operand whose
// slots hold a multiple of 64 rows does the same from the mapped first row of
// the stage; any other split operand resolves every k-row through RowSrc.  The
// two arms issue textually different copies
// (dma16<1> for the split one): with identical ones the compiler sinks the copy
// below the branch and computes both addresses on every copy.
struct Mn2Rows {
  uint32_t off0;   // element offset of the lane's 16 bytes for copy 0 at k0 = 0
};

template <int WAVES>
__device__ __forceinline__ Mn2Rows mn2_rows(const Operand& op, int x0, int wave, int lane) {
  const int kr = 2 * wave + (lane >> 5);
  const int lc = (lane & 31) ^ mn_swz(kr);
  int x = x0 + lc * 8;
  if (x >= op.rows) x = op.rows - 8;
  return Mn2Rows{static_cast<uint32_t>(kr * op.src.ld + x)};
}

template <int WAVES>
__device__ __forceinline__ void copy2_mn(uint8_t* lds, const Operand& op, const Mn2Rows& rows, int x0, int k0,
                                         int wave, int lane) {
  // A stage's 64 k-rows are consecutive in memory when the operand is one
  // plain array, and also when it is split but every sequence-parallel slot
  // holds a multiple of 64 rows (stages start at multiples of 64, so none
  // straddles a slot or a sequence): then the stage's first row is mapped
  // once (uniform, scalar) and each lane adds its fixed offset.
  if (op.src.t == 1 || op.src.s_sp % BK2 == 0) {       // uniform
    const uint16_t* base0;
    if (op.src.t == 1) {
      base0 = op.src.own + static_cast<int64_t>(k0) * op.src.ld;
    } else {
      // pick own or peer by arithmetic on the two pointer values: a select of
      // the members' addresses would put the kernel argument on the stack
      const uint32_t o = op.src.row_index(k0);
      const uint64_t own = reinterpret_cast<uint64_t>(op.src.own), peer = reinterpret_cast<uint64_t>(op.src.peer);
      const uint64_t pick = own + ((peer - own) & (0ull - static_cast<uint64_t>(o >> 31)));
      base0 = reinterpret_cast<const uint16_t*>(pick) + static_cast<int64_t>(o & 0x7fffffffu) * op.src.ld;
    }
#pragma unroll
    for (int q = 0; q < 32 / WAVES; ++q)
      dma16(base0 + static_cast<int64_t>(2 * WAVES * q) * op.src.ld + rows.off0, lds + (wave + WAVES * q) * 1024);
    return;
  }
#pragma unroll
  for (int q = 0; q < 32 / WAVES; ++q) {
    const int kb = wave + WAVES * q;
    const int kr = 2 * kb + (lane >> 5);
    const int lc = (lane & 31) ^ mn_swz(kr);
    int x = x0 + lc * 8;
    if (x >= op.rows) x = op.rows - 8;
    const uint32_t o = op.src.row_index(k0 + kr);
    const uint16_t* base = (o & 0x80000000u) ? op.src.peer : op.src.own;
    dma16<1>(base + static_cast<int64_t>(o & 0x7fffffffu) * op.src.ld + x, lds + kb * 1024);
  }
}

template <int NS>
struct Frags2 {
  bf16x8 a[4], b[NS];
};

// KC fragment of rows x0 + lane%32 (x0 a multiple of 32), k = 16 kk + 8 (lane/32) + 0..7.
template <Layout L>
__device__ __forceinline__ bf16x8 frag2(const uint8_t* lds, int x0, int kk, int lane) {
  if constexpr (L == Layout::KC) {
    return *reinterpret_cast<const bf16x8*>(lds + kc2_off(x0 + (lane & 31), 2 * kk + (lane >> 5)));
  } else {
    return frag<Layout::MN>(lds, x0, kk, lane);
  }
}

// Fragments are read in the order the products consume them (A0, B0 .. B(NS-1),
// A1, A2, A3), so the first products of the next sub-step wait on the
// earliest reads.
template <Layout LA, Layout LB, int NS>
__device__ __forceinline__ void read_frags2(Frags2<NS>& f, const uint8_t* la, const uint8_t* lb, int wm,
                                            const int* ncol, int kk, int lane) {
  f.a[0] = frag2<LA>(la, wm * 128, kk, lane);
#pragma unroll
  for (int ns = 0; ns < NS; ++ns) f.b[ns] = frag2<LB>(lb, ncol[ns], kk, lane);
#pragma unroll
  for (int ms = 1; ms < 4; ++ms) f.a[ms] = frag2<LA>(la, wm * 128 + ms * 32, kk, lane);
}

template <int NS>
__device__ __forceinline__ void mfma_frags2(f32x16 (&acc)[4][NS], const Frags2<NS>& f) {
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int ns = 0; ns < NS; ++ns)
      acc[ms][ns] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[ms], f.b[ns], acc[ms][ns], 0, 0, 0);
}

// Spread DS reads over the MFMAs of a sub-step: 8 slots of (DS share, M MFMAs).
// A K-contiguous fragment is one LDS read, a transposed one two.
template <int DS, int M, int I = 0>
__device__ __forceinline__ void interleave2_slots() {
  if constexpr (I < 8) {
    constexpr int n = (DS * (I + 1)) / 8 - (DS * I) / 8;
    if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(0x100, n, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, M, 0);
    interleave2_slots<DS, M, I + 1>();
  }
}
template <Layout LA, Layout LB, int NS>
__device__ __forceinline__ void interleave2() {
  constexpr int DS = 4 * (LA == Layout::KC ? 1 : 2) + NS * (LB == Layout::KC ? 1 : 2);
  interleave2_slots<DS, NS / 2>();
}

// The BK = 64 main loop of one tile over its stages [kb, kb + n), n even:
// products added into acc.  The four stage buffers a0 b0 a1 b1 (32 KB each)
// hold two stages.
template <Layout LA, Layout LB, int WAVES>
__device__ __forceinline__ void mainloop64(const GemmParams& p, f32x16 (&acc)[4][WAVES == 8 ? 2 : 4], int tm, int tn,
                                           int kb, int n, uint8_t* a0, uint8_t* b0, uint8_t* a1, uint8_t* b1,
                                           int wave, int lane, int wm, const int* ncol) {
  constexpr int NS = WAVES == 8 ? 2 : 4;
  constexpr int PER = 32 / WAVES;           // copy instructions per operand per stage per wave
  const int m0 = tm * BM, n0 = tn * BN;
  Kc2Rows<WAVES> ra{}, rb{};
  Mn2Rows ma{}, mb{};
  if constexpr (LA == Layout::KC) ra = kc2_rows<WAVES>(p.A, m0, tm, wave, lane);
  else ma = mn2_rows<WAVES>(p.A, m0, wave, lane);
  if constexpr (LB == Layout::KC) rb = kc2_rows<WAVES>(p.B, n0, tn, wave, lane);
  else mb = mn2_rows<WAVES>(p.B, n0, wave, lane);
  // stage kt of the range (stages past its end repeat the last one: the wait counts stay fixed)
  auto issue_a = [&](int kt, uint8_t* la) {
    const int k0 = (kb + min(kt, n - 1)) * BK2;
    if constexpr (LA == Layout::KC) copy2_kc<WAVES>(la, ra, k0, wave);
    else copy2_mn<WAVES>(la, p.A, ma, m0, k0, wave, lane);
  };
  auto issue_b = [&](int kt, uint8_t* lb) {
    const int k0 = (kb + min(kt, n - 1)) * BK2;
    if constexpr (LB == Layout::KC) copy2_kc<WAVES>(lb, rb, k0, wave);
    else copy2_mn<WAVES>(lb, p.B, mb, n0, k0, wave, lane);
  };

  Frags2<NS> f0, f1;
  // Stage kt (buffers X, next stage in Y): sub-steps kk = 0..3 each read the
  // fragments of the next sub-step under their own MFMAs.  Before the last
  // sub-step every wave has read all of X: wait for stage kt+1, publish it
  // with the barrier, refill X's A half with stage kt+2 and read the first
  // fragments of Y under the last MFMAs.  The B half of stage kt+2 follows at
  // the start of stage kt+1 (measured a few percent faster than issuing both
  // halves at the barrier).
  auto stage = [&](int kt, uint8_t* xa, uint8_t* xb, const uint8_t* ya, uint8_t* yb) {
    if (kt > 0) {
      issue_b(kt + 1, yb);   // stage kt+1's B half (Y's B buffer was freed at kt-1's barrier)
      __builtin_amdgcn_sched_barrier(0);
    }
    read_frags2<LA, LB, NS>(f1, xa, xb, wm, ncol, 1, lane);
    mfma_frags2<NS>(acc, f0);
    interleave2<LA, LB, NS>();
    read_frags2<LA, LB, NS>(f0, xa, xb, wm, ncol, 2, lane);
    mfma_frags2<NS>(acc, f1);
    interleave2<LA, LB, NS>();
    read_frags2<LA, LB, NS>(f1, xa, xb, wm, ncol, 3, lane);
    mfma_frags2<NS>(acc, f0);
    interleave2<LA, LB, NS>();
    wait_vm<0>();
    stage_barrier();
    issue_a(kt + 2, xa);
    // Keep the copies here, right after the barrier: left alone, the scheduler
    // sinks them to the end of the next stage, next to the wait for them, and
    // no computation overlaps their latency.
    __builtin_amdgcn_sched_barrier(0);
    read_frags2<LA, LB, NS>(f0, ya, yb, wm, ncol, 0, lane);   // after the last stage: read, never used
    mfma_frags2<NS>(acc, f1);
    interleave2<LA, LB, NS>();
  };

  issue_a(0, a0);
  issue_b(0, b0);
  issue_a(1, a1);
  issue_b(1, b1);
  if constexpr (PER == 8) wait_vm<16>();
  else wait_vm<8>();
  stage_barrier();
  read_frags2<LA, LB, NS>(f0, a0, b0, wm, ncol, 0, lane);
  for (int kt = 0; kt < n; kt += 2) {
    stage(kt, a0, b0, a1, b1);
    stage(kt + 1, a1, b1, a0, b0);
  }
  wait_vm<0>();      // the last (repeated) stage copy has landed
}

// Wave-private staging space of the epilogue in the stage buffers.
template <int WAVES>
__device__ __forceinline__ float* stage_space(uint8_t* a0, uint8_t* b0, uint8_t* a1, uint8_t* b1, int wave) {
  const int q = WAVES == 8 ? (wave >> 1) : wave;
  uint8_t* mine = q == 0 ? a0 : q == 1 ? b0 : q == 2 ? a1 : b1;
  if constexpr (WAVES == 8) mine += (wave & 1) * 16384;
  return reinterpret_cast<float*>(mine);
}

template <Layout LA, Layout LB, EpiKind KIND, int PAIR, int WAVES>
__global__ void __launch_bounds__(WAVES * 64, 1) gemm_bk64(GemmParams p) {
  constexpr int NS = WAVES == 8 ? 2 : 4;
  __shared__ __attribute__((aligned(16))) uint8_t a0[TILE2], b0[TILE2], a1[TILE2], b1[TILE2];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave: scalar code for wave-level decisions
  // AccF32 with a split K range: the grid is k_splits copies of the tile grid,
  // part-major after the XCD remap, so an XCD's neighbouring tiles share a part.
  constexpr bool kSplittable = KIND == EpiKind::AccF32 || KIND == EpiKind::StoreBF16;
  const int parts = kSplittable && p.k_splits > 1 ? p.k_splits : 1;
  const int pid_all = xcd_remap(blockIdx.x, gridDim.x);
  const int tiles = static_cast<int>(gridDim.x) / parts;
  const int part = pid_all / tiles;
  const TileCoord tc = tile_coord(p, pid_all - part * tiles);
  const int tm = tc.tm, tn = tc.tn, m0 = tm * BM;
  const int wm = WAVES == 8 ? (wave >> 2) : (wave >> 1);
  const int wn = WAVES == 8 ? (wave & 3) : (wave & 1);
  int ncol[NS];
#pragma unroll
  for (int j = 0; j < NS / 2; ++j) {
    ncol[j] = lo_col<WAVES, PAIR>(wn, j);
    ncol[j + NS / 2] = ncol[j] + PAIR;
  }
  const int n_st = p.K / BK2 / parts;          // stages per part (the host keeps it even)
  float* cbase = nullptr;
  int64_t ldc = 0;
  if constexpr (KIND == EpiKind::AccF32) {
    cbase = part == 0 ? static_cast<float*>(p.epi.c) : p.partial + static_cast<int64_t>(part - 1) * p.M * p.N;
    ldc = part == 0 ? p.epi.ldc : p.N;
  } else if constexpr (KIND == EpiKind::StoreBF16) {
    // split: every part stores its fp32 sum; the reduce pass adds them and rounds to bf16
    cbase = p.partial + static_cast<int64_t>(part) * p.M * p.N;
    ldc = p.N;
  }

  f32x16 acc[4][NS];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[i][j] = f32x16{};
  // K is a multiple of 2 * BK2 * parts (the host picks this kernel only then).
  mainloop64<LA, LB, WAVES>(p, acc, tm, tn, part * n_st, n_st, a0, b0, a1, b1, wave, lane, wm, ncol);
  // The fp32 accumulate: the products start from zero and part 0 adds the C
  // tile in the epilogue, whose loads overlap its stores (loading C into the
  // accumulators before the first product measured 2-3% slower on the largest
  // weight-gradient GEMMs of the Llama-3-70B TP8 shard).
  if (KIND == EpiKind::AccF32 && part == 0) {
    acc_add_store_f32<NS>(acc, p, cbase, ldc, static_cast<int64_t>(m0) + wm * 128, tn, ncol, lane);
    return;
  }
  if (KIND == EpiKind::AccF32 || (KIND == EpiKind::StoreBF16 && parts > 1)) {
    acc_store_f32<NS>(acc, p, cbase, ldc, static_cast<int64_t>(m0) + wm * 128, tn, ncol, lane);
  } else {
    __syncthreads();   // every wave is done reading the stages
    store_tile<KIND, PAIR, NS>(p, acc, stage_space<WAVES>(a0, b0, a1, b1, wave), static_cast<int64_t>(m0) + wm * 128,
                               tn, ncol, lane);
  }
}

// Kernel choice: K a multiple of 128 (and every K split) takes the 8-wave
// BK = 64 kernel, the fastest on the Llama layer shapes; any other K the
// BK = 32 kernel, whose copies mask the ragged end of K.
template <Layout LA, Layout LB, EpiKind KIND, int PAIR>
hipError_t launch(const GemmParams& p, hipStream_t stream) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.B.split_rows ? (p.B.split_rows + 127) / 128 : (p.N + BN - 1) / BN;
  const int parts = p.k_splits > 1 ? p.k_splits : 1;
  if (parts > 1 && ((KIND != EpiKind::AccF32 && KIND != EpiKind::StoreBF16) || p.K % (2 * BK2 * parts) != 0 ||
                    !p.partial))
    return hipErrorInvalidValue;
  // the fp32 accumulate's whole-tile epilogue addresses 128 rows of C with 32-bit byte offsets
  if (KIND == EpiKind::AccF32 && p.epi.ldc > (int64_t{1} << 21)) return hipErrorInvalidValue;
  const dim3 grid(tiles_m * tiles_n * parts);
  if (p.K % (2 * BK2) == 0)
    hipLaunchKernelGGL((gemm_bk64<LA, LB, KIND, PAIR, 8>), grid, dim3(512), 0, stream, p);
  else
    hipLaunchKernelGGL((gemm_bk32<LA, LB, KIND, PAIR>), grid, dim3(512), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm(const GemmParams& p, Layout la, Layout lb, hipStream_t stream) {
  if (p.M <= 0 || p.N <= 0 || p.K <= 0) return hipSuccess;
  using L = Layout;
  using E = EpiKind;
  const E k = p.epi.kind;
  if (la == L::KC && lb == L::KC) {
    if (k == E::QkvRope && p.epi.d_h == 128) return launch<L::KC, L::KC, E::QkvRope, 64>(p, stream);
    if (k == E::QkvRope && p.epi.d_h == 64) return launch<L::KC, L::KC, E::QkvRope, 32>(p, stream);
    if (k == E::ResidualSP) return launch<L::KC, L::KC, E::ResidualSP, 128>(p, stream);
    if (k == E::SwiGLUFwd) return launch<L::KC, L::KC, E::SwiGLUFwd, 128>(p, stream);
    if (k == E::StoreBF16) return launch<L::KC, L::KC, E::StoreBF16, 128>(p, stream);
    if (k == E::StoreF32) return launch<L::KC, L::KC, E::StoreF32, 128>(p, stream);
  } else if (la == L::KC && lb == L::MN) {
    if (k == E::SwiGLUBwd) return launch<L::KC, L::MN, E::SwiGLUBwd, 128>(p, stream);
    if (k == E::ResidualSP) return launch<L::KC, L::MN, E::ResidualSP, 128>(p, stream);
    if (k == E::StoreBF16) return launch<L::KC, L::MN, E::StoreBF16, 128>(p, stream);
    if (k == E::StoreF32) return launch<L::KC, L::MN, E::StoreF32, 128>(p, stream);
    if (k == E::AccF32) return launch<L::KC, L::MN, E::AccF32, 128>(p, stream);
  } else if (la == L::MN && lb == L::MN) {
    if (k == E::AccF32) return launch<L::MN, L::MN, E::AccF32, 128>(p, stream);
  }
  return hipErrorInvalidValue;     // a layout / epilogue pairing the layer never uses
}

namespace {
// C += partial[0] + partial[1] + ..., four floats per thread (N % 4 == 0 and
// ldc % 4 == 0 are required by the caller).
__global__ void __launch_bounds__(256) split_reduce_kernel(float* __restrict__ c, int64_t ldc,
                                                          const float* __restrict__ part, int64_t M, int64_t N,
                                                          int32_t n_part) {
  const int64_t n4 = N / 4;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= M * n4) return;
  const int64_t m = i / n4, j = (i - m * n4) * 4;
  float4* cp = reinterpret_cast<float4*>(c + m * ldc + j);
  float4 v = *cp;
  for (int s = 0; s < n_part; ++s) {
    const float4 q = *reinterpret_cast<const float4*>(part + static_cast<int64_t>(s) * M * N + m * N + j);
    v.x += q.x;
    v.y += q.y;
    v.z += q.z;
    v.w += q.w;
  }
  *cp = v;
}
// C (bf16) = partial[0] + partial[1] + ..., four columns per thread.
__global__ void __launch_bounds__(256) split_store_kernel(uint16_t* __restrict__ c, int64_t ldc,
                                                         const float* __restrict__ part, int64_t M, int64_t N,
                                                         int32_t n_part) {
  const int64_t n4 = N / 4;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= M * n4) return;
  const int64_t m = i / n4, j = (i - m * n4) * 4;
  float4 v = *reinterpret_cast<const float4*>(part + m * N + j);
  for (int s = 1; s < n_part; ++s) {
    const float4 q = *reinterpret_cast<const float4*>(part + static_cast<int64_t>(s) * M * N + m * N + j);
    v.x += q.x;
    v.y += q.y;
    v.z += q.z;
    v.w += q.w;
  }
  uint16_t* o = c + m * ldc + j;
  o[0] = f2bf(v.x);
  o[1] = f2bf(v.y);
  o[2] = f2bf(v.z);
  o[3] = f2bf(v.w);
}
}  // namespace

hipError_t gemm_split_store(uint16_t* c, int64_t ldc, const float* partial, int64_t M, int64_t N, int32_t splits,
                            hipStream_t stream) {
  if (splits < 1 || M <= 0 || N <= 0) return hipSuccess;
  const int64_t n = M * (N / 4);
  hipLaunchKernelGGL(split_store_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, c, ldc,
                     partial, M, N, splits);
  return hipGetLastError();
}

int gemm_ksplits(int64_t M, int64_t N, int64_t K, bool acc_f32) {
  // Model: a wave of 256 tiles of full K takes T = 2*256*256*K / (1 PFLOP/s / 256 CUs);
  // s parts take ceil(tiles*s / 256) waves of T/s, plus writing and reading the
  // fp32 partials at about 4 TB/s (s - 1 of them when part 0 accumulates into an
  // fp32 C, all s when the result is stored as bf16).  Pick the cheapest s of 1..4.
  // The rate is deliberately low: the chip is power-limited, so a wave that
  // leaves CUs idle runs at a higher clock than tile counting suggests (the
  // 160-tile qkv weight gradient of the 70B shard was no faster in 4 parts),
  // and only clearly under-filled grids (128 tiles) split.
  const int64_t tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const double t_wave = 2.0 * BM * BN * static_cast<double>(K) / (1e15 / 256.0);
  int best = 1;
  double best_t = 1e30;
  for (int s = 1; s <= 4; ++s) {
    if (K % (2 * BK2 * s) != 0 || N % 4 != 0) continue;
    const double waves = static_cast<double>((tiles * s + 255) / 256);
    const int n_part = s == 1 ? 0 : (acc_f32 ? s - 1 : s);
    const double t = waves * t_wave / s + n_part * 2.0 * 4.0 * static_cast<double>(M) * N / 4e12;
    if (t < best_t * 0.97) {       // a split has to win by a margin
      best_t = t;
      best = s;
    }
  }
  return best;
}

hipError_t gemm_split_reduce(float* c, int64_t ldc, const float* partial, int64_t M, int64_t N, int32_t splits,
                             hipStream_t stream) {
  if (splits <= 1 || M <= 0 || N <= 0) return hipSuccess;
  const int64_t n = M * (N / 4);
  hipLaunchKernelGGL(split_reduce_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, c, ldc,
                     partial, M, N, splits - 1);
  return hipGetLastError();
}

}  // namespace l4d
