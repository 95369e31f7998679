// Causal grouped-query attention on the gfx950 matrix cores, FlashAttention
// style: the forward keeps only the output and the per-row log-sum-exp, the
// backward recomputes the probabilities from Q, K and the log-sum-exp
// (the activation accounting of Sec. 3.2 counts QK^T and softmax as zero).
//
// Keys come as up to kMaxSeg runs with consecutive global positions: the
// rank's own context-parallel chunks and the remote chunks of the other CP
// ranks.  A key is visible to a query iff key position <= query position.
//
// gfx950 design:
//  * every K/V/Q/dO tile is copied global -> LDS with global_load_lds_dwordx4
//    (no staging registers) into a row-major tile with an XOR swizzle of its
//    16-byte chunks; two separate LDS buffers alternate so that the next tile
//    streams in while the current one is used;
//  * operands that need the token index contiguous (V in P V, Q and dO in the
//    dK/dV products, K in dQ) are read transposed straight from those tiles
//    with ds_read_b64_tr_b16 (16 lanes x 4 rows -> 4 rows per lane);
//  * scores are computed transposed where that puts one query per lane
//    (forward, dQ), so the softmax statistics are per-lane scalars; the bf16
//    probabilities then feed the next MFMA from registers with the
//    contraction index permuted consistently on both operands;
//  * masks are applied only on tiles that straddle the diagonal;
//  * 256 threads and 64 KB of LDS per workgroup: two workgroups per CU.
//  * dK/dV are accumulated over the query heads of a kv-head inside one
//    workgroup, or, when that leaves too few workgroups, over a slice of them
//    with an fp32 partial per slice that a small kernel sums: no atomics, the
//    result is deterministic.
#include <math.h>

#include <type_traits>

#include <algorithm>
#include <vector>

#include "kernels.h"

namespace l4d {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

#define LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int KT = 64;            // keys per tile (forward, dQ)
constexpr int QT = 64;            // queries per tile (dK/dV)
// LDS fragment reads kept in flight ahead of the products, per kernel
constexpr int kLookFwd = 6, kLookDq = 4, kLookDkv = 4;

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// Two floats to a packed bf16 pair with one conversion (round to nearest even).
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}
__device__ __forceinline__ float lo16(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi16(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// Wait until at most N of this wave's copies are still in flight.
template <int N>
__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }
// Workgroup barrier that does not drain the copies still in flight (unlike
// __syncthreads): only this wave's LDS reads must be done before it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Make the compiler wait for a value loaded from global memory here, before
// the tile loop: otherwise it places the wait at the value's first use inside
// the loop, on every iteration, where the hardware counter also holds the
// next tile's copies (issued as inline assembly) -- and the wait drains them.
template <class T>
__device__ __forceinline__ void settle(const T& v) {
  asm volatile("" ::"v"(v));
}

// ------------------------------------------------------------------ LDS tiles
// Row-major [rows][D] bf16 tile; 16-byte chunk c of row r sits at chunk c ^ swz(r).
// The LDS serves 256 bytes (64 banks) per cycle.  Two read patterns must be
// conflict-free: a row fragment (16 lanes, 16 consecutive rows, one chunk
// each) needs swz to be a permutation over every aligned block of 16 rows; a
// transposing column fragment (32 lanes, 4 consecutive rows x an aligned group
// of 4 chunks) needs the 4 rows to map that group to 4 different groups, i.e.
// distinct swz >> 2 across 4 consecutive rows.  At D = 64 a row is half a
// bank line, so row parity picks the half and swz only has to separate rows
// of equal parity.  Also swz(r + 8) = swz(r) ^ 4: a column fragment reads
// rows r and r + 8, and the second address is then the first address of the
// neighbouring 32-column block plus a constant, so no extra register holds it.
template <int D>
__device__ __forceinline__ int swz(int row) {
  const int b1 = (row >> 1) & 1, b2 = (row >> 2) & 1, b3 = (row >> 3) & 1;
  return D == 128 ? ((((row & 3) ^ b3) << 2) | (b2 << 1) | (row & 1)) : (((b1 ^ b3) << 2) | (b2 << 1) | b1);
}

// Direct-to-LDS copy of `size` bytes per lane from sbase + voff (uniform base,
// per-lane byte offset) into the wave's LDS chunk at lds (lane i lands at
// lds + size * i).  Inline assembly: the compiler's wait-count pass does not
// see the LDS write in flight, so it does not drain the prefetch before the
// reads of the other buffer (it cannot tell the buffers apart).  The kernels
// wait for their own copies (vmcnt) before the barrier that publishes a tile.
// The LDS address is uniform by construction; readfirstlane states it for the
// compiler, which otherwise may keep it in a vector register.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, const uint8_t* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(LPTR(const_cast<uint8_t*>(lds)))));
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(l) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* sbase, uint32_t voff, const void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>(LPTR(const_cast<void*>(lds)))));
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(sbase), "s"(l) : "memory", "m0");
}

// Copy rows [0, ROWS) of src (row stride ld, rows >= n_valid clamped to the
// last valid row) into an LDS tile; the NW waves of the block share the work.
// A copy instruction moves RPK whole rows (1 KB); lane i lands at byte 16 i of
// the instruction's LDS chunk.  The wave's copies start at rows that agree
// modulo 4 * RPK (the waves take every NW-th chunk, NW a multiple of 4), which
// fixes swz, so each lane's swizzled source column is fixed: the row block is
// a uniform base and the lane adds one 32-bit byte offset, except on a ragged tail.
template <int D, int ROWS, int NW = 4>
__device__ __forceinline__ void tile_load(uint8_t* lds, const uint16_t* src, int64_t ld, int n_valid, int wave,
                                          int lane) {
  constexpr int CH = D / 8;              // 16-byte chunks per row
  constexpr int RPK = 64 / CH;           // rows per 1 KB wave chunk
  constexpr int NKB = ROWS / RPK;
  static_assert(NKB % NW == 0, "every wave issues the same number of copies");
  const int lrow = lane / CH;
  const int lc = (lane % CH) ^ swz<D>(wave * RPK + lrow);   // the same for every copy of this wave
  const int ldb = static_cast<int>(ld) * 2;                 // row stride in bytes
  if (n_valid >= ROWS) {
    const uint32_t lane_off = static_cast<uint32_t>(lrow * ldb + lc * 16);
#pragma unroll
    for (int j = 0; j < NKB / NW; ++j) {
      const int q = wave + j * NW;
      dma16(src + static_cast<int64_t>(q * RPK) * ld, lane_off, lds + q * 1024);
    }
  } else {                               // ragged tail: rows past n_valid repeat the last valid row
#pragma unroll
    for (int j = 0; j < NKB / NW; ++j) {
      const int q = wave + j * NW;
      const int r = min(q * RPK + lrow, n_valid - 1);
      dma16(src, static_cast<uint32_t>(r * ldb + lc * 16), lds + q * 1024);
    }
  }
}

// Per-lane LDS byte offsets of the two fragment shapes below, at kk = 0 and
// dt = 0 of a tile's first row block.  With swz periodic in 16 rows, the
// other kk / dt are an XOR of the low byte (the 16-byte chunk within a row),
// and other row blocks a constant: one register per shape.
struct LaneAddr {
  int rows;   // row fragment: row lane%32, chunk lane/32
  int cols;   // column fragment: row 4 (lane/32) + (lane%16)/4, column 16 ((lane/16)%2) + 4 (lane%4)
};
template <int D>
__device__ __forceinline__ LaneAddr lane_addr(int lane) {
  const int h = lane >> 5, li = lane & 15;
  const int rr = lane & 31;
  const int cr = 4 * h + (li >> 2);
  const int low = 2 * ((lane >> 4) & 1) + ((li & 3) >> 1);   // chunk within the 4-chunk group
  return LaneAddr{rr * (D * 2) + ((swz<D>(rr) ^ h) << 4),
                  cr * (D * 2) + ((low ^ swz<D>(cr)) << 4) + ((li & 1) << 3)};
}
// MFMA operand with the tile's rows as its 32 rows: rows row0 + lane%32 (row0
// a multiple of 16), contraction chunk 2*kk + lane/32 (d = 16 kk + 8 (lane/32) + 0..7).
template <int D>
__device__ __forceinline__ bf16x8 frag_rows(const uint8_t* lds, int row0, int kk, LaneAddr la) {
  return *reinterpret_cast<const bf16x8*>(lds + row0 * (D * 2) + (la.rows ^ (kk << 5)));
}
// MFMA operand with the tile's columns as its rows: d = 32 dt + lane%32; its 8
// contraction slots are tile rows 16 g16 + {4h .. 4h+3, 8+4h .. 8+4h+3},
// h = lane/32 -- the same order in which a lane holds accumulator rows of a
// 32x32 MFMA (see frag_acc).  Two transposing 64-bit LDS reads; rows r + 8
// have swz(r) ^ 4, which is the XOR pattern of column block dt ^ 1.
template <int D>
__device__ __forceinline__ bf16x8 frag_cols(const uint8_t* lds, int dt, int g16, LaneAddr la) {
  const uint8_t* base = lds + g16 * 16 * (D * 2);
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<__attribute__((address_space(3))) i16x4*>(
      LPTR(const_cast<uint8_t*>(base) + (la.cols ^ (dt << 6)))));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(reinterpret_cast<__attribute__((address_space(3))) i16x4*>(
      LPTR(const_cast<uint8_t*>(base) + 8 * (D * 2) + (la.cols ^ ((dt ^ 1) << 6)))));
  return __builtin_bit_cast(bf16x8, u32x4{__builtin_bit_cast(u32x2, a)[0], __builtin_bit_cast(u32x2, a)[1],
                                          __builtin_bit_cast(u32x2, b)[0], __builtin_bit_cast(u32x2, b)[1]});
}
// Operand from 8 accumulator registers i0..i0+7 (rows 16 (i0/8) + {4h..4h+3, 8+4h..}).
__device__ __forceinline__ bf16x8 frag_acc(const f32x16& s, int i0) {
  return __builtin_bit_cast(bf16x8, u32x4{pack2(s[i0], s[i0 + 1]), pack2(s[i0 + 2], s[i0 + 3]),
                                          pack2(s[i0 + 4], s[i0 + 5]), pack2(s[i0 + 6], s[i0 + 7])});
}
// The rounding residual of frag_acc: bf16(s - hi) for the same 8 registers,
// given hi = frag_acc(s, i0).  hi + lo carries about 16 significant bits.
__device__ __forceinline__ bf16x8 frag_acc_lo(const f32x16& s, int i0, bf16x8 hi) {
  const u32x4 h = __builtin_bit_cast(u32x4, hi);
  u32x4 r;
#pragma unroll
  for (int k = 0; k < 4; ++k) r[k] = pack2(s[i0 + 2 * k] - lo16(h[k]), s[i0 + 2 * k + 1] - hi16(h[k]));
  return __builtin_bit_cast(bf16x8, r);
}
// Row of accumulator register i for this lane (32x32 MFMA output layout).
__device__ __forceinline__ int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// Global position of local query row `row` (at most two chunks).  A select
// between the two scalar chunk ids, not an indexed load: a per-lane index into
// the kernel arguments would become a vector load whose wait drains every copy
// in flight.
__device__ __forceinline__ int qpos(const ChunkMap& m, int row) {
  const bool second = row >= m.chunk_len;
  return (second ? m.chunk_id[1] : m.chunk_id[0]) * m.chunk_len + (second ? row - m.chunk_len : row);
}

// Key tile `tile` (of `tsz` tokens) across the segments.
__device__ __forceinline__ bool find_tile(const AttnParams& p, int tile, int tsz, int& seg, int& t0) {
  int acc = 0;
  for (int s = 0; s < p.n_seg; ++s) {
    const int nt = (p.seg[s].n + tsz - 1) / tsz;
    if (tile < acc + nt) {
      seg = s;
      t0 = (tile - acc) * tsz;
      return true;
    }
    acc += nt;
  }
  return false;
}

// ------------------------------------------------------------------ forward
// One workgroup per (128-query tile, query head, batch element); 4 waves x 32
// queries, each lane holding one query's scores (S^T = K Q^T).  The launch is
// one-dimensional with the head index varying fastest and the query tiles in
// descending order, so the longest causal rows are dispatched first across all
// heads.  Registers stay within 256 per lane and LDS within 64 KB, so two
// workgroups share a CU and each SIMD interleaves the matrix products of one
// wave with the softmax of another.
//
// The output and the row sum are rescaled only on tiles where some row's
// maximum grew (a wave-wide vote).  The reference maximum stays exact: a
// stale one would leave the largest probability of a row off the bf16 grid
// point 1 and, for sharply peaked rows, double the rounding error of ctx.

// Next key tile to visit at or after (seg, t0): the first tile of a segment
// whose first key a query at pos_max can see.  Positions grow within a
// segment, so the rest of a segment is skipped once a tile starts past pos_max.
__device__ __forceinline__ bool next_tile(const AttnParams& p, int pos_max, int& seg, int& t0) {
  while (seg < p.n_seg) {
    if (t0 < p.seg[seg].n && p.seg[seg].pos0 + t0 <= pos_max) return true;
    ++seg;
    t0 = 0;
  }
  return false;
}

// Two-stage copy ring over the key tiles of `step` keys that a query at
// pos_max can see: tile j is computed from buffer j % 2 while tile j + 1 lands
// in the other.  `issue(seg, t0, buf)` starts a tile's copies, `compute(seg,
// t0, buf)` uses it; buf is std::integral_constant<int, 0 or 1>, so every LDS
// object is named statically and the compiler sees that reads of one buffer
// do not depend on the copies landing in the other.
template <class Issue, class Compute>
__device__ __forceinline__ void run_ring2(const AttnParams& p, int pos_max, int step, Issue issue, Compute compute) {
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  int cs = 0, ct = 0;
  bool have = next_tile(p, pos_max, cs, ct);
  if (have) issue(cs, ct, B0{});
  while (have) {
    int ns = cs, nt = ct + step;
    bool more = next_tile(p, pos_max, ns, nt);
    wait_copies<0>();
    ring_barrier();                      // every wave's copy is visible; the other buffer is free
    if (more) issue(ns, nt, B1{});
    __builtin_amdgcn_sched_barrier(0);   // the copies go out now, not next to the wait for them
    compute(cs, ct, B0{});
    if (!more) break;
    cs = ns;
    ct = nt;
    ns = cs;
    nt = ct + step;
    more = next_tile(p, pos_max, ns, nt);
    wait_copies<0>();
    ring_barrier();
    if (more) issue(ns, nt, B0{});
    __builtin_amdgcn_sched_barrier(0);
    compute(cs, ct, B1{});
    have = more;
    cs = ns;
    ct = nt;
  }
}

// ------------------------------------------------------------------ pipelined products
// Two accumulator chains over the D columns of LDS tiles, with the B operands
// in registers:  s0 += A0[r0 + (0..31)] x0^T,  s1 += A1[r1 + (0..31)] x1^T.
// The schedule keeps LA fragment reads in flight ahead of the products
// (without it the compiler reads each fragment right before its product and
// the LDS latency is exposed on every step).
template <int D, int LA>
__device__ __forceinline__ void scores2(const uint8_t* a0, int r0, const bf16x8 (&x0)[D / 16], f32x16& s0,
                                        const uint8_t* a1, int r1, const bf16x8 (&x1)[D / 16], f32x16& s1,
                                        LaneAddr la) {
  constexpr int N = D / 8;               // products (and fragment reads)
  constexpr int L = LA < N ? LA : N - 1;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    s0 = mfma(frag_rows<D>(a0, r0, kk, la), x0[kk], s0);
    s1 = mfma(frag_rows<D>(a1, r1, kk, la), x1[kk], s1);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, L, 0);      // LDS reads
#pragma unroll
  for (int i = 0; i < N - L; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, L, 0);
}

// acc[dt] += A^T x over NG groups of 16 rows: A the LDS tile read transposed
// (d rows, row-index contraction), x[g] a bf16 operand from registers (P^T,
// dS^T); two reads per fragment, LA fragments in flight.
template <int D, int NG, int LA>
__device__ __forceinline__ void accum_t(const uint8_t* lds, const bf16x8 (&x)[NG], f32x16 (&acc)[D / 32], LaneAddr la) {
  constexpr int N = NG * D / 32;
  constexpr int L = LA < N ? LA : N - 1;
#pragma unroll
  for (int g = 0; g < NG; ++g)
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = mfma(frag_cols<D>(lds, dt, g, la), x[g], acc[dt]);
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * L, 0);
#pragma unroll
  for (int i = 0; i < N - L; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, L, 0);
}

// acc[dt] += A^T (xh + xl): as accum_t with the register operand split into a
// high and a low bf16 part; each transposed fragment feeds both products, and
// the high products of a group's column blocks go before their low products,
// so no product waits on the one just before it.
template <int D, int NG, int LA>
__device__ __forceinline__ void accum_t2(const uint8_t* lds, const bf16x8 (&xh)[NG], const bf16x8 (&xl)[NG],
                                         f32x16 (&acc)[D / 32], LaneAddr la) {
  constexpr int N = NG * D / 32;
  constexpr int L = LA < N ? LA : N - 1;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    bf16x8 f[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) f[dt] = frag_cols<D>(lds, dt, g, la);
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = mfma(f[dt], xh[g], acc[dt]);
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] = mfma(f[dt], xl[g], acc[dt]);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * L, 0);
#pragma unroll
  for (int i = 0; i < N - L; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2 * L, 0);
}

template <int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) attn_fwd_kernel(AttnParams p) {
  constexpr int TB = KT * D * 2;
  __shared__ __attribute__((aligned(16))) uint8_t k0[TB], v0[TB], k1[TB], v1[TB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_qt = (p.n_q + 127) / 128;
  const int nh = p.a_t * p.b;
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.x) / nh;   // heaviest tiles first
  const int hq = static_cast<int>(blockIdx.x) % nh % p.a_t, bi = static_cast<int>(blockIdx.x) % nh / p.a_t;
  const int hk = hq / (p.a_t / p.k_t);
  const int q_row0 = qt * 128;
  const int my_q = q_row0 + wave * 32 + (lane & 31);
  const bool q_ok = my_q < p.n_q;
  const int my_pos = q_ok ? qpos(p.qmap, my_q) : -1;
  const int blk_last = min(q_row0 + 127, p.n_q - 1);
  const int pos_min = qpos(p.qmap, q_row0), pos_max = qpos(p.qmap, blk_last);
  const int rbase = 4 * (lane >> 5);
  const LaneAddr la = lane_addr<D>(lane);

  bf16x8 qf[D / 16];
  {
    const uint16_t* qb = p.q + bi * p.q_bstride + static_cast<int64_t>(q_ok ? my_q : 0) * p.q_ld + hq * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qb + (2 * kk + (lane >> 5)) * 8);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) settle(qf[kk]);
  }
  const float c = p.scale * kLog2e;
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) o[i] = f32x16{};

  auto issue = [&](int seg, int t0, uint8_t* kt, uint8_t* vt) __attribute__((always_inline)) {
    const KvSeg& s = p.seg[seg];
    const int64_t off = bi * s.bstride + static_cast<int64_t>(t0) * s.ld + hk * D;
    tile_load<D, KT>(kt, s.k + off, s.ld, s.n - t0, wave, lane);
    tile_load<D, KT>(vt, s.v + off, s.ld, s.n - t0, wave, lane);
  };
  auto compute = [&](int seg, int t0, const uint8_t* kt, const uint8_t* vt) __attribute__((always_inline)) {
    const int kpos0 = p.seg[seg].pos0 + t0;
    const int kvalid = min(KT, p.seg[seg].n - t0);
    f32x16 sc[2] = {f32x16{}, f32x16{}};
    scores2<D, kLookFwd>(kt, 0, qf, sc[0], kt, 32, qf, sc[1], la);
    if (kpos0 + KT - 1 > pos_min || kvalid < KT) {       // tile straddles the diagonal (or is ragged)
      // last visible key row for this query, relative to the lane's first row
      const int lim = min(my_pos - kpos0, kvalid - 1) - rbase;
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (t2 * 32 + 8 * (i >> 2) + (i & 3) > lim) sc[t2][i] = -INFINITY;
    }
    float mx = __builtin_fmaxf(sc[0][0], sc[0][1]);           // a chain of three-input maxima
#pragma unroll
    for (int i = 2; i < 16; i += 2) mx = __builtin_fmaxf(__builtin_fmaxf(mx, sc[0][i]), sc[0][i + 1]);
#pragma unroll
    for (int i = 0; i < 16; i += 2) mx = __builtin_fmaxf(__builtin_fmaxf(mx, sc[1][i]), sc[1][i + 1]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c;
    if (__builtin_amdgcn_ballot_w64(mx > m_run)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);   // 0 while m_run is -inf
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) o[dt] *= alpha;
      l_run *= alpha;
      m_run = m_new;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    float rs = 0.f;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pr = fast_exp2(fmaf(sc[t2][i], c, -m_use));
        sc[t2][i] = pr;
        rs += pr;
      }
    l_run += rs;
    // P enters the P V product as bf16 hi + lo parts (two products per V
    // fragment): a plain bf16 P carries a relative error of up to 2^-9 into
    // every output, which the bf16 stores after attention then amplify.
    bf16x8 pf[4], pl[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      pf[g] = frag_acc(sc[g >> 1], 8 * (g & 1));
      pl[g] = frag_acc_lo(sc[g >> 1], 8 * (g & 1), pf[g]);
    }
    accum_t2<D, 4, kLookFwd>(vt, pf, pl, o, la);
  };

  run_ring2(
      p, pos_max, KT,
      [&](int seg, int t0, auto b) __attribute__((always_inline)) {
        if constexpr (decltype(b)::value == 0) issue(seg, t0, k0, v0);
        else issue(seg, t0, k1, v1);
      },
      [&](int seg, int t0, auto b) __attribute__((always_inline)) {
        if constexpr (decltype(b)::value == 0) compute(seg, t0, k0, v0);
        else compute(seg, t0, k1, v1);
      });

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!q_ok) return;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  uint16_t* ob = p.o + bi * p.q_bstride + static_cast<int64_t>(my_q) * p.q_ld + hq * D;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + rbase;
      *reinterpret_cast<u32x2*>(ob + d) = u32x2{pack2(o[dt][4 * jj] * inv, o[dt][4 * jj + 1] * inv),
                                                pack2(o[dt][4 * jj + 2] * inv, o[dt][4 * jj + 3] * inv)};
    }
  if (lane < 32) {
    const float m_fin = m_run == -INFINITY ? 0.f : m_run;
    p.lse[(static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q + my_q] = (m_fin + __builtin_amdgcn_logf(l_tot)) * kLn2;
  }
}


// ------------------------------------------------------------------ backward: dK, dV
// Flat grid over (key block of 128 over all segments, kv head, split, b), key
// block slowest: the earliest key blocks see the most query tiles, so they are
// dispatched first (longest job first keeps the last CUs from running one long
// block alone), and with the heads varying fastest every block of a head lands
// on the same XCD (dispatch deals block ids round-robin over the 8 XCDs),
// where its query-tile stream is shared in L2.  8 waves.
// Workgroup (kb, hk, split) sums over query heads hk*g + [split*hpb, (split+1)*hpb).
//
// The block's 128 keys form four groups of 32, and each group has two waves
// with different jobs, on the same SIMD (wave w runs on SIMD w % 4):
//  * role 0 (waves 0-3) holds K, computes S^T = K Q^T, P^T = exp(S^T - lse),
//    hands P^T (fp32) to its partner through LDS and accumulates dV^T += dO^T P^T;
//  * role 1 (waves 4-7) holds V, computes dP^T = V dO^T, takes P^T and forms
//    dS^T = P^T (dP^T - delta), and accumulates dK^T += Q^T dS^T.
// Each wave then needs one operand block and one accumulator block, which fits
// 256 registers, and the two waves of a SIMD issue different instruction mixes
// (softmax on one, products on the other) that interleave.  dS^T is formed
// from the fp32 P^T and rounded to bf16 once, as in the dQ kernel.
template <int D>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2))) attn_bwd_dkdv_kernel(AttnParams p) {
  constexpr int TB = QT * D * 2;
  // Two stages of Q and dO tiles (64 KB at D = 128: every tile offset fits a
  // ds_read immediate), then the statistics and the P^T handover.
  __shared__ __attribute__((aligned(16))) uint8_t qg0[2][TB], qg1[2][TB];   // per stage: Q tile, then dO tile
  __shared__ __attribute__((aligned(16))) float st0[2][QT], st1[2][QT];             // lse, delta
  // P^T handover in fp32, so that dS^T = P^T (dP^T - delta) rounds once: [group][16 queries][half][lane]
  __shared__ __attribute__((aligned(16))) float4 xp[4][QT / 16][2][64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave & 3, role = wave >> 2;
  const int group = p.a_t / p.k_t;
  const int hpb = group / p.n_split;
  const int nyz = p.k_t * p.n_split * p.b;
  const int kb_raw = static_cast<int>(blockIdx.x) / nyz, yz = static_cast<int>(blockIdx.x) % nyz;
  const int kb = p.n_order ? p.kb_order[kb_raw] : kb_raw;
  const int hk = yz % (p.k_t * p.n_split) / p.n_split, split = yz % p.n_split;
  const int bi = yz / (p.k_t * p.n_split);
  int seg, k0;
  if (!find_tile(p, kb, 128, seg, k0)) return;
  const KvSeg& S = p.seg[seg];
  const int my_key = k0 + grp * 32 + (lane & 31);
  const bool key_ok = my_key < S.n;
  const int my_kpos = S.pos0 + my_key;
  const int grp_kpos0 = S.pos0 + k0 + grp * 32;
  const int blk_kpos0 = S.pos0 + k0;
  const int rbase = 4 * (lane >> 5);
  const LaneAddr la = lane_addr<D>(lane);
  // Offsets into a stage's [Q | dO] pair: the first product reads Q (role 0)
  // or dO (role 1), the second reads dO (role 0) or Q (role 1).
  const LaneAddr la1{la.rows + role * TB, la.cols};
  const LaneAddr la2{la.rows, la.cols + (1 - role) * TB};

  bf16x8 kv[D / 16];                     // role 0: K rows, role 1: V rows of the group's keys
  {
    const uint16_t* src = role == 0 ? S.k : S.v;
    const int64_t off = bi * S.bstride + static_cast<int64_t>(key_ok ? my_key : 0) * S.ld + hk * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      kv[kk] = *reinterpret_cast<const bf16x8*>(src + off + (2 * kk + (lane >> 5)) * 8);
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) settle(kv[kk]);
  }
  f32x16 acc[D / 32];                    // role 0: dV^T, role 1: dK^T (d rows, the lane's key)
#pragma unroll
  for (int i = 0; i < D / 32; ++i) acc[i] = f32x16{};
  const float c = p.scale * kLog2e;
  const int n_qt = (p.n_q + QT - 1) / QT;
  const int total = hpb * n_qt;
  const int head0 = hk * group + split * hpb;
  auto next_wanted = [&](int from) __attribute__((always_inline)) {
    for (int it = from; it < total; ++it) {
      const int qt = it % n_qt;
      const int last = min(qt * QT + QT - 1, p.n_q - 1);
      if (qpos(p.qmap, last) >= blk_kpos0) return it;
    }
    return total;
  };
  auto issue = [&](int it, uint8_t* qt_l, uint8_t* gt_l, float (*st)[QT]) __attribute__((always_inline)) {
    const int hq = head0 + it / n_qt, qt = it % n_qt;
    if (lane < 16) {    // waves 0-3 copy the lse, waves 4-7 delta, of queries 16 grp .. 16 grp + 15
      const int q = min(qt * QT + grp * 16 + lane, p.n_q - 1);
      const float* row = (role == 0 ? p.lse : p.delta) + (static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q;
      dma4(row, static_cast<uint32_t>(q) * 4u, &st[role][grp * 16]);
    }
    const int64_t off = bi * p.q_bstride + static_cast<int64_t>(qt * QT) * p.q_ld + hq * D;
    tile_load<D, QT, 8>(qt_l, p.q + off, p.q_ld, p.n_q - qt * QT, wave, lane);
    tile_load<D, QT, 8>(gt_l, p.dout + off, p.q_ld, p.n_q - qt * QT, wave, lane);
  };
  // One query tile (64 queries as four 16-query groups g; MFMA halves h = g / 2).
  auto compute = [&](int it, const uint8_t* qt_l, const uint8_t* gt_l, const float (*st)[QT]) __attribute__((always_inline)) {
    const int qt = it % n_qt;
    const int qr0 = qt * QT;
    const int qlast = min(qr0 + QT - 1, p.n_q - 1);
    const int qp0 = qpos(p.qmap, qr0), qpl = qpos(p.qmap, qlast);
    // Every group works on every tile the block visits; on the one or two
    // diagonal tiles where all of a group's keys follow every query, the
    // causal mask zeroes its P^T (a skip there would cost register copies at
    // the branch joins on every tile).
    const bool full = qp0 >= grp_kpos0 + 31 && qlast == qr0 + QT - 1 && qpl - qp0 == QT - 1;
    const bool contiguous = qpl - qp0 == qlast - qr0;
    // Both roles run one instruction stream over role-selected tiles (role 0:
    // S^T from Q, dV^T from dO; role 1: dP^T from dO, dK^T from Q), so the
    // accumulators never meet at a branch join.
    f32x16 s[2] = {f32x16{}, f32x16{}};              // role 0: S^T -> P^T, role 1: dP^T -> dS^T
    bf16x8 x[4];                                       // role 0: P^T, role 1: dS^T (bf16)
    scores2<D, kLookDkv>(qt_l, 0, kv, s[0], qt_l, 32, kv, s[1], la1);
    {
      if (role == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const float4 ls = *reinterpret_cast<const float4*>(&st[0][32 * h + 8 * jj + rbase]);
            const float lsv[4] = {ls.x * kLog2e, ls.y * kLog2e, ls.z * kLog2e, ls.w * kLog2e};
#pragma unroll
            for (int u = 0; u < 4; ++u) s[h][4 * jj + u] = fast_exp2(fmaf(s[h][4 * jj + u], c, -lsv[u]));
          }
        if (!full) {                                   // causal / ragged masks
          if (contiguous) {
            // visible query rows r (relative to the lane's first row): lo <= r <= hi
            const int lo = (key_ok ? my_kpos - qp0 : QT) - rbase;
            const int hi = qlast - qr0 - rbase;
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
              for (int i = 0; i < 16; ++i) {
                const int r = 32 * h + 8 * (i >> 2) + (i & 3);
                if (r < lo || r > hi) s[h][i] = 0.f;
              }
          } else {                                     // the tile spans two context-parallel chunks
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
              for (int i = 0; i < 16; ++i) {
                const int qr = 32 * h + 8 * (i >> 2) + rbase + (i & 3);
                const int qp = qr0 + qr <= qlast ? qpos(p.qmap, qr0 + qr) : -1;
                if (my_kpos > qp || !key_ok) s[h][i] = 0.f;
              }
          }
        }
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int h = g >> 1, i0 = 8 * (g & 1);
          x[g] = frag_acc(s[h], i0);                   // bf16 P^T for this wave's dV product
          xp[grp][g][0][lane] = make_float4(s[h][i0], s[h][i0 + 1], s[h][i0 + 2], s[h][i0 + 3]);
          xp[grp][g][1][lane] = make_float4(s[h][i0 + 4], s[h][i0 + 5], s[h][i0 + 6], s[h][i0 + 7]);
        }
      }
    }
    ring_barrier();                                    // P^T of every group is visible to its partner
    if (role == 1) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 p0 = xp[grp][g][0][lane], p1 = xp[grp][g][1][lane];
        const float pv[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
        const int h = g >> 1, i0 = 8 * (g & 1);
        const float4 d0 = *reinterpret_cast<const float4*>(&st[1][32 * h + (i0 >> 2) * 8 + rbase]);
        const float4 d1 = *reinterpret_cast<const float4*>(&st[1][32 * h + ((i0 >> 2) + 1) * 8 + rbase]);
        const float dev[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
        float ds[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) ds[j] = pv[j] * (s[h][i0 + j] - dev[j]);
        x[g] = __builtin_bit_cast(
            bf16x8, u32x4{pack2(ds[0], ds[1]), pack2(ds[2], ds[3]), pack2(ds[4], ds[5]), pack2(ds[6], ds[7])});
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    accum_t<D, 4, kLookDkv>(qt_l, x, acc, la2);
  };

  // Two-stage ring over the query tiles: tile j is used from one buffer set
  // while tile j + 1 lands in the other.
  int cur = next_wanted(0);
  if (cur < total) issue(cur, qg0[0], qg0[1], st0);
  while (cur < total) {
    int nxt = next_wanted(cur + 1);
    wait_copies<0>();
    ring_barrier();                      // tile cur is visible; the other buffers are free
    if (nxt < total) issue(nxt, qg1[0], qg1[1], st1);
    __builtin_amdgcn_sched_barrier(0);   // the copies go out now, not next to the wait for them
    compute(cur, qg0[0], qg0[1], st0);
    if (nxt >= total) break;
    cur = nxt;
    nxt = next_wanted(cur + 1);
    wait_copies<0>();
    ring_barrier();
    if (nxt < total) issue(nxt, qg0[0], qg0[1], st0);
    __builtin_amdgcn_sched_barrier(0);
    compute(cur, qg1[0], qg1[1], st1);
    cur = nxt;
  }

  if (!key_ok) return;
  // lane owns key my_key; register i of tile dt is d = 32 dt + acc_row(i)
  if (role == 1) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) acc[dt] *= p.scale;
  }
  if (p.n_split > 1) {
    // fp32 partial [split][b][key (over segments)][k_t][D], dK then dV at +partial_half; summed by attn_dkv_reduce
    const int64_t key_index = static_cast<int64_t>(p.seg_key0[seg]) + my_key;
    const int64_t row = ((static_cast<int64_t>(split) * p.b + bi) * p.total_keys + key_index) * p.k_t + hk;
    float* pa = p.dkv_partial + (role == 1 ? 0 : p.partial_half) + row * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d = dt * 32 + 8 * jj + rbase;
        *reinterpret_cast<float4*>(pa + d) = make_float4(acc[dt][4 * jj], acc[dt][4 * jj + 1], acc[dt][4 * jj + 2],
                                                         acc[dt][4 * jj + 3]);
      }
    return;
  }
  const int64_t off = bi * S.bstride + static_cast<int64_t>(my_key) * S.ld + hk * D;
  const int64_t doff = bi * S.d_bstride + static_cast<int64_t>(my_key) * S.d_ld + hk * D;
  const uint16_t* receipt = role == 1 ? S.rk : S.rv;
  if (receipt) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d = dt * 32 + 8 * jj + rbase;
        const u32x2 r = *reinterpret_cast<const u32x2*>(receipt + off + d);
        acc[dt][4 * jj] += lo16(r[0]);
        acc[dt][4 * jj + 1] += hi16(r[0]);
        acc[dt][4 * jj + 2] += lo16(r[1]);
        acc[dt][4 * jj + 3] += hi16(r[1]);
      }
  }
  if (role == 1 && S.rope) {
    constexpr int HALF_T = D / 64;
    const float2* tab = p.rope + static_cast<int64_t>(S.rope_row0 + my_key) * (D / 2);
#pragma unroll
    for (int dt = 0; dt < HALF_T; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float2 cs = tab[dt * 32 + acc_row(i, lane)];
        const float a = acc[dt][i], b = acc[dt + HALF_T][i];
        acc[dt][i] = a * cs.x + b * cs.y;              // rotate by -angle
        acc[dt + HALF_T][i] = b * cs.x - a * cs.y;
      }
  }
  uint16_t* dst = (role == 1 ? S.dk : S.dv) + doff;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + rbase;
      *reinterpret_cast<u32x2*>(dst + d) =
          u32x2{pack2(acc[dt][4 * jj], acc[dt][4 * jj + 1]), pack2(acc[dt][4 * jj + 2], acc[dt][4 * jj + 3])};
    }
}

// Sum the per-slice fp32 partials, add the receipts, apply the inverse RoPE to
// local keys and store bf16.  One 64-thread block per (key, kv-head, b); thread
// j handles the RoPE pair (j, j + D/2) of dK and of dV.
template <int D>
__global__ void __launch_bounds__(64) attn_dkv_reduce_kernel(AttnParams p) {
  const int key_index = blockIdx.x, hk = blockIdx.y, bi = blockIdx.z;
  const int j = threadIdx.x;
  if (j >= D / 2) return;
  int seg = 0;
  while (seg + 1 < p.n_seg && key_index >= p.seg_key0[seg + 1]) ++seg;
  const KvSeg& S = p.seg[seg];
  const int key = key_index - p.seg_key0[seg];
  float a = 0.f, b = 0.f, va = 0.f, vb = 0.f;
  for (int sp = 0; sp < p.n_split; ++sp) {
    const int64_t row = ((static_cast<int64_t>(sp) * p.b + bi) * p.total_keys + key_index) * p.k_t + hk;
    const float* pk = p.dkv_partial + row * D;
    const float* pv = p.dkv_partial + p.partial_half + row * D;
    a += pk[j];
    b += pk[j + D / 2];
    va += pv[j];
    vb += pv[j + D / 2];
  }
  const int64_t off = bi * S.bstride + static_cast<int64_t>(key) * S.ld + hk * D;
  if (S.rk) {
    a += __uint_as_float(static_cast<uint32_t>(S.rk[off + j]) << 16);
    b += __uint_as_float(static_cast<uint32_t>(S.rk[off + j + D / 2]) << 16);
    va += __uint_as_float(static_cast<uint32_t>(S.rv[off + j]) << 16);
    vb += __uint_as_float(static_cast<uint32_t>(S.rv[off + j + D / 2]) << 16);
  }
  if (S.rope) {
    const float2 cs = p.rope[static_cast<int64_t>(S.rope_row0 + key) * (D / 2) + j];
    const float ra = a * cs.x + b * cs.y, rb = b * cs.x - a * cs.y;
    a = ra;
    b = rb;
  }
  const int64_t doff = bi * S.d_bstride + static_cast<int64_t>(key) * S.d_ld + hk * D;
  S.dk[doff + j] = f2bf(a);
  S.dk[doff + j + D / 2] = f2bf(b);
  S.dv[doff + j] = f2bf(va);
  S.dv[doff + j + D / 2] = f2bf(vb);
}

// ------------------------------------------------------------------ backward: dQ
// One workgroup per (128-query tile, query head, batch element), flat grid in
// the forward's heaviest-first order; 4 waves x 32 queries.  Key tiles of 32
// keep Q, dO, dQ and the two score tiles within 256 registers, so two
// workgroups share a CU.  Per tile: S^T = K Q^T and dP^T = V dO^T, then
// dS^T = P^T (dP^T - delta) feeds dQ^T += K^T dS^T from registers.
// delta = rowsum(dO * O) of the block's queries is formed here, from the dO
// fragments it holds anyway and the matching fragments of O, and written out
// for the dK/dV pass, which runs after this one.
template <int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) attn_bwd_dq_kernel(AttnParams p) {
  constexpr int KQ = 32;                     // keys per tile
  constexpr int TB = KQ * D * 2;
  __shared__ __attribute__((aligned(16))) uint8_t k0[TB], v0[TB], k1[TB], v1[TB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_qt = (p.n_q + 127) / 128;
  const int nh = p.a_t * p.b;
  const int qt = n_qt - 1 - static_cast<int>(blockIdx.x) / nh;
  const int hq = static_cast<int>(blockIdx.x) % nh % p.a_t, bi = static_cast<int>(blockIdx.x) % nh / p.a_t;
  const int hk = hq / (p.a_t / p.k_t);
  const int q_row0 = qt * 128;
  const int my_q = q_row0 + wave * 32 + (lane & 31);
  const bool q_ok = my_q < p.n_q;
  const int my_pos = q_ok ? qpos(p.qmap, my_q) : -1;
  const int blk_last = min(q_row0 + 127, p.n_q - 1);
  const int pos_min = qpos(p.qmap, q_row0), pos_max = qpos(p.qmap, blk_last);
  const int rbase = 4 * (lane >> 5);
  const LaneAddr la = lane_addr<D>(lane);

  bf16x8 qf[D / 16], dof[D / 16];
  float my_delta = 0.f;
  {
    const int64_t off = bi * p.q_bstride + static_cast<int64_t>(q_ok ? my_q : 0) * p.q_ld + hq * D;
    u32x4 of[D / 16];
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const int dcol = (2 * kk + (lane >> 5)) * 8;
      qf[kk] = *reinterpret_cast<const bf16x8*>(p.q + off + dcol);
      dof[kk] = *reinterpret_cast<const bf16x8*>(p.dout + off + dcol);
      of[kk] = *reinterpret_cast<const u32x4*>(p.o + off + dcol);
    }
    // the lane's half of the row (8-column chunks of one parity), then its partner's half
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const u32x4 g = __builtin_bit_cast(u32x4, dof[kk]);
#pragma unroll
      for (int j = 0; j < 4; ++j) my_delta += lo16(g[j]) * lo16(of[kk][j]) + hi16(g[j]) * hi16(of[kk][j]);
    }
    my_delta += __shfl_xor(my_delta, 32, 64);
  }
  const int64_t sidx = (static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q + (q_ok ? my_q : 0);
  const float my_lse = p.lse[sidx] * kLog2e;
  if (q_ok && lane < 32) p.delta[sidx] = my_delta;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    settle(qf[kk]);
    settle(dof[kk]);
  }
  settle(my_lse);
  settle(my_delta);
  const float c = p.scale * kLog2e;
  f32x16 dq[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dq[i] = f32x16{};

  auto issue = [&](int seg, int t0, uint8_t* kt, uint8_t* vt) __attribute__((always_inline)) {
    const KvSeg& s = p.seg[seg];
    const int64_t off = bi * s.bstride + static_cast<int64_t>(t0) * s.ld + hk * D;
    tile_load<D, KQ>(kt, s.k + off, s.ld, s.n - t0, wave, lane);
    tile_load<D, KQ>(vt, s.v + off, s.ld, s.n - t0, wave, lane);
  };
  auto compute = [&](int seg, int t0, const uint8_t* kt, const uint8_t* vt) __attribute__((always_inline)) {
    const int kpos0 = p.seg[seg].pos0 + t0;
    const int kvalid = min(KQ, p.seg[seg].n - t0);
    f32x16 sc = f32x16{}, dp = f32x16{};
    scores2<D, kLookDq>(kt, 0, qf, sc, vt, 0, dof, dp, la);
    if (kpos0 + KQ - 1 > pos_min || kvalid < KQ) {      // tile straddles the diagonal (or is ragged)
      const int lim = (q_ok ? min(my_pos - kpos0, kvalid - 1) : -1) - rbase;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (8 * (i >> 2) + (i & 3) > lim) sc[i] = -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) sc[i] = fast_exp2(fmaf(sc[i], c, -my_lse)) * (dp[i] - my_delta);   // dS^T
    const bf16x8 sf[2] = {frag_acc(sc, 0), frag_acc(sc, 8)};
    accum_t<D, 2, kLookDq>(kt, sf, dq, la);
  };
  run_ring2(
      p, pos_max, KQ,
      [&](int seg, int t0, auto b) __attribute__((always_inline)) {
        if constexpr (decltype(b)::value == 0) issue(seg, t0, k0, v0);
        else issue(seg, t0, k1, v1);
      },
      [&](int seg, int t0, auto b) __attribute__((always_inline)) {
        if constexpr (decltype(b)::value == 0) compute(seg, t0, k0, v0);
        else compute(seg, t0, k1, v1);
      });

  if (!q_ok) return;
  constexpr int HALF_T = D / 64;
  const float2* tab = p.rope + static_cast<int64_t>(my_q) * (D / 2);
#pragma unroll
  for (int dt = 0; dt < HALF_T; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float2 cs = tab[dt * 32 + acc_row(i, lane)];
      const float a = dq[dt][i] * p.scale, b = dq[dt + HALF_T][i] * p.scale;
      dq[dt][i] = a * cs.x + b * cs.y;
      dq[dt + HALF_T][i] = b * cs.x - a * cs.y;
    }
  uint16_t* out = p.dq + (bi * static_cast<int64_t>(p.n_q) + my_q) * p.dq_ld + hq * D;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + rbase;
      *reinterpret_cast<u32x2*>(out + d) =
          u32x2{pack2(dq[dt][4 * jj], dq[dt][4 * jj + 1]), pack2(dq[dt][4 * jj + 2], dq[dt][4 * jj + 3])};
    }
}

int count_blocks(const AttnParams& p, int tsz) {
  int n = 0;
  for (int s = 0; s < p.n_seg; ++s) n += (p.seg[s].n + tsz - 1) / tsz;
  return n;
}

template <int D>
hipError_t fwd_impl(const AttnParams& p, hipStream_t stream) {
  const unsigned blocks = static_cast<unsigned>((p.n_q + 127) / 128) * p.a_t * p.b;
  hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3(blocks), dim3(256), 0, stream, p);
  return hipGetLastError();
}

// Host copy of the query-tile walk of the dK/dV kernel: the number of 64-query
// tiles a 128-key block starting at global position kpos0 visits per head.
int dkdv_tiles(const AttnParams& p, int kpos0) {
  const int n_qt = (p.n_q + QT - 1) / QT;
  int n = 0;
  for (int qt = 0; qt < n_qt; ++qt) {
    const int last = std::min(qt * QT + QT - 1, p.n_q - 1);
    const bool second = last >= p.qmap.chunk_len;
    const int pos = (second ? p.qmap.chunk_id[1] : p.qmap.chunk_id[0]) * p.qmap.chunk_len +
                    (second ? last - p.qmap.chunk_len : last);
    if (pos >= kpos0) ++n;
  }
  return n;
}

// Dispatch order of the dK/dV key blocks: most query tiles first (stable), so
// that with context parallelism the long blocks of every key segment start
// before the short ones instead of segment by segment.
void dkdv_order(AttnParams& p) {
  const int nb = count_blocks(p, 128);
  p.n_order = 0;
  if (nb > kMaxKeyBlocks) return;
  std::vector<std::pair<int, int>> w;
  w.reserve(nb);
  int kb = 0;
  for (int s = 0; s < p.n_seg; ++s)
    for (int k0 = 0; k0 < p.seg[s].n; k0 += 128, ++kb) w.push_back({-dkdv_tiles(p, p.seg[s].pos0 + k0), kb});
  std::stable_sort(w.begin(), w.end(), [](const auto& a, const auto& b) { return a.first < b.first; });
  for (int i = 0; i < nb; ++i) p.kb_order[i] = static_cast<uint16_t>(w[i].second);
  p.n_order = nb;
}

template <int D>
hipError_t bwd_impl(const AttnParams& p, int part, hipStream_t stream) {
  if (part == 1) {
    const unsigned blocks = static_cast<unsigned>(count_blocks(p, 128)) * p.k_t * p.n_split * p.b;
    AttnParams q = p;
    dkdv_order(q);
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<D>, dim3(blocks), dim3(512), 0, stream, q);
  } else if (part == 3) {
    if (p.n_split == 1) return hipSuccess;
    hipLaunchKernelGGL(attn_dkv_reduce_kernel<D>, dim3(p.total_keys, p.k_t, p.b), dim3(64), 0, stream, p);
  } else {
    const unsigned blocks = static_cast<unsigned>((p.n_q + 127) / 128) * p.a_t * p.b;
    hipLaunchKernelGGL(attn_bwd_dq_kernel<D>, dim3(blocks), dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace

int attn_bwd_splits(const AttnParams& p) {
  // Split the query heads of a kv-head over workgroups until the dK/dV grid
  // has at least 512 workgroups (two per CU) or every head has its own.
  const int group = p.a_t / p.k_t;
  const int base = count_blocks(p, 128) * p.k_t * p.b;
  int n = 1;
  while (base * n < 512 && n < group && group % (2 * n) == 0) n *= 2;
  return n;
}

hipError_t attn_fwd(const AttnParams& p, hipStream_t stream) {
  if (p.n_q <= 0) return hipSuccess;
  if (p.d_h == 128) return fwd_impl<128>(p, stream);
  if (p.d_h == 64) return fwd_impl<64>(p, stream);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd(const AttnParams& p, int part, hipStream_t stream) {
  if (p.n_q <= 0) return hipSuccess;
  if (p.d_h == 128) return bwd_impl<128>(p, part, stream);
  if (p.d_h == 64) return bwd_impl<64>(p, part, stream);
  return hipErrorInvalidValue;
}

}  // namespace l4d
