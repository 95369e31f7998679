// bf16 GEMM on the gfx950 matrix cores: C[m][n] = sum_k A(m,k) B(n,k), fp32
// accumulation, with the layer's fused epilogues.
//
// Tiling: a 512-thread workgroup (8 waves, two per SIMD) owns a 256x256 tile
// of C; each wave accumulates a 128x64 block as 4 x 2 tiles of
// v_mfma_f32_32x32x16_bf16 (128 accumulator registers).  K advances in steps
// of 32 through a 4-stage pipeline: operand tiles are copied global -> LDS by
// global_load_lds_dwordx4 (one contiguous KB per wave instruction, no staging
// registers) three steps ahead of their use.  Every stage buffer is its own
// LDS object so the compiler knows a read of one stage cannot depend on the
// copies still landing in the others.
//
// Operand layouts: "KC" (reduction index contiguous: activations in the
// forward, the output gradient in dX) is stored as two 16-k sub-blocks of
// 256 rows x 32 bytes, the two halves of a row swapped on rows with bit 2
// set: the 8 rows one fragment read touches fall in 8 different bank groups
// and every fragment address is a per-lane base plus an immediate.  "MN"
// (reduction index strided: the weight in dX, both operands of dW) is stored
// as 32 k-rows x 256 columns with the 16-byte chunks XOR-swizzled by row, and
// read with two ds_read_b64_tr_b16 that hand each lane 4 consecutive k of one
// column -- the transpose happens in the LDS read, not in registers.
//
// A wave's two 32-column blocks sit PAIR columns apart, so the columns n and
// n + PAIR land in the same lane and register: a RoPE pair (i, i + d_h/2) or a
// gate/up pair of the fused FFN weight.  The epilogue stages 64 rows at a time
// through LDS and hands 8-column vectors to the fused operation.
#include <stdlib.h>

#include "kernels.h"

namespace l4d {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define GPTR(p) ((const __attribute__((address_space(1))) void*)(p))
#define LPTR(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int BM = 256, BN = 256, BK = 32;
constexpr int TILE_BYTES = 256 * BK * 2;     // 16 KB per operand per stage
constexpr int GROUP_M = 8;

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ u32x4 pack8(const float* v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = (uint32_t)f2bf(v[2 * i]) | ((uint32_t)f2bf(v[2 * i + 1]) << 16);
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
// KC tile: 16-byte chunk c (0..3) of row r (0..255) in sub-block c/2.
__device__ __forceinline__ int kc_off(int row, int chunk) {
  return (chunk >> 1) * 8192 + row * 32 + (((chunk & 1) ^ ((row >> 2) & 1)) << 4);
}
// MN tile: k-row r (0..31), 16-byte chunk c (0..31) of its 256 columns.
__device__ __forceinline__ int mn_swz(int row) { return (row & 3) << 1; }
__device__ __forceinline__ int mn_off(int row, int chunk) { return row * 512 + ((chunk ^ mn_swz(row)) << 4); }

// Each stage holds 16 KB per operand; wave w copies LDS KB numbers
// kb = w + WAVES * q.  KC: KB kb holds sub-block kb/8 and tile rows
// 32 * (kb % 8) + lane/2, so a lane's source rows are fixed over K; they are
// kept as 32-bit element offsets, bit 31 selecting the peer base of a
// sequence-parallel gather.  MN: KB kb holds k-rows 2 kb + lane/32.
template <int WAVES>
struct KcRows {
  uint32_t off[8 / WAVES];   // one per distinct row block kb % 8 of this wave
};

template <int WAVES>
__device__ __forceinline__ KcRows<WAVES> kc_rows(const Operand& op, int x0, int tile_idx, int wave, int lane) {
  KcRows<WAVES> r;
#pragma unroll
  for (int j = 0; j < 8 / WAVES; ++j) {
    const int xr = 32 * (wave + WAVES * j) + (lane >> 1);
    int64_t gx;
    if (op.split_rows) {
      int i = tile_idx * 128 + (xr & 127);
      if (i >= op.split_rows) i = op.split_rows - 1;
      gx = (xr >= 128 ? op.split_off : 0) + i;
    } else {
      gx = x0 + xr;
      if (gx >= op.rows) gx = op.rows - 1;
    }
    r.off[j] = op.src.row_index(gx);
  }
  return r;
}

template <int WAVES>
__device__ __forceinline__ void copy_kc(uint8_t* lds, const Operand& op, const KcRows<WAVES>& rows, int k0, int K,
                                        int wave, int lane) {
#pragma unroll
  for (int q = 0; q < 16 / WAVES; ++q) {
    const int kb = wave + WAVES * q;
    const int kk = kb >> 3;
    const int row = 32 * (kb & 7) + (lane >> 1);
    const uint32_t o = rows.off[q % (8 / WAVES)];
    const uint16_t* base = ((o & 0x80000000u) ? op.src.peer : op.src.own) +
                           static_cast<int64_t>(o & 0x7fffffffu) * op.src.ld;
    const int hh = (lane & 1) ^ ((row >> 2) & 1);
    int k = k0 + kk * 16 + hh * 8;
    if (k >= K) k = K - 8;            // those fragments are zeroed before use
    __builtin_amdgcn_global_load_lds(GPTR(base + k), LPTR(lds + kb * 1024), 16, 0, 0);
  }
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
    __builtin_amdgcn_global_load_lds(GPTR(base + static_cast<int64_t>(o & 0x7fffffffu) * op.src.ld + x),
                                     LPTR(lds + kb * 1024), 16, 0, 0);
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

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// lo: 8 columns starting at tile column `col`; hi: the 8 columns PAIR further.
template <EpiKind KIND, int PAIR>
__device__ __forceinline__ void epilogue(const GemmParams& p, int64_t m, int tn, int col, float* lo, float* hi) {
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
    case EpiKind::AccF32: {
      float* c = static_cast<float*>(e.c) + m * e.ldc;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = n_lo + h * PAIR;
        const float* src = h ? hi : lo;
        if (n < p.N) {
          float4* d = reinterpret_cast<float4*>(c + n);
          float4 a = d[0], b = d[1];
          a.x += src[0]; a.y += src[1]; a.z += src[2]; a.w += src[3];
          b.x += src[4]; b.y += src[5]; b.z += src[6]; b.w += src[7];
          d[0] = a;
          d[1] = b;
        }
      }
      break;
    }
    case EpiKind::QkvRope: {
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
        const int32_t i = static_cast<int32_t>(m % e.s_c);
        const float2* tab = e.rope + static_cast<int64_t>(i) * (e.d_h / 2) + (n % e.d_h);
        float a[8], b[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float2 cs = tab[j];
          a[j] = lo[j] * cs.x - hi[j] * cs.y;
          b[j] = hi[j] * cs.x + lo[j] * cs.y;
        }
        *reinterpret_cast<u32x4*>(dst + m * ld + n) = pack8(a);
        *reinterpret_cast<u32x4*>(dst + m * ld + n + PAIR) = pack8(b);
      } else {
        *reinterpret_cast<u32x4*>(dst + m * ld + n) = pack8(lo);
        *reinterpret_cast<u32x4*>(dst + m * ld + n + PAIR) = pack8(hi);
      }
      break;
    }
    case EpiKind::ResidualSP: {
      int64_t orow = m;
      bool own = true;
      if (e.t > 1) {
        const int64_t bi = m / e.s_c;
        const int32_t i = static_cast<int32_t>(m - bi * e.s_c);
        const int32_t lo_row = e.r * e.s_sp;
        own = i >= lo_row && i < lo_row + e.s_sp;
        orow = own ? bi * e.s_sp + (i - lo_row)
                   : bi * static_cast<int64_t>(e.t - 1) * e.s_sp + (i < lo_row ? i : i - e.s_sp);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = n_lo + h * PAIR;
        if (n >= p.N) continue;
        float* src = h ? hi : lo;
        const int64_t off = orow * e.ldc + n;
        if (own) {
          float r[8];
          if (e.resid) {
            unpack8(*reinterpret_cast<const u32x4*>(e.resid + off), r);
#pragma unroll
            for (int j = 0; j < 8; ++j) src[j] += r[j];
          }
          if (e.receipt) {
            unpack8(*reinterpret_cast<const u32x4*>(e.receipt + off), r);
#pragma unroll
            for (int j = 0; j < 8; ++j) src[j] += r[j];
          }
          *reinterpret_cast<u32x4*>(e.own_out + off) = pack8(src);
        } else {
          *reinterpret_cast<u32x4*>(e.send + off) = pack8(src);
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
        a[q] = silu_f(g[q]);
        pr[q] = a[q] * u[q];
      }
      *reinterpret_cast<u32x4*>(e.g_out + off) = pack8(g);
      *reinterpret_cast<u32x4*>(e.u_out + off) = pack8(u);
      *reinterpret_cast<u32x4*>(e.act_out + off) = pack8(a);
      *reinterpret_cast<u32x4*>(e.prod_out + off) = pack8(pr);
      break;
    }
    case EpiKind::SwiGLUBwd: {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = n_lo + h * PAIR;
        if (n >= p.N) continue;
        const float* dp = h ? hi : lo;
        const int64_t off = m * e.f + n;
        float g[8], u[8], a[8], dg[8], du[8];
        unpack8(*reinterpret_cast<const u32x4*>(e.g_in + off), g);
        unpack8(*reinterpret_cast<const u32x4*>(e.u_in + off), u);
        unpack8(*reinterpret_cast<const u32x4*>(e.act_in + off), a);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const float s = 1.0f / (1.0f + __expf(-g[q]));
          dg[q] = dp[q] * u[q] * (s * (1.0f + g[q] * (1.0f - s)));
          du[q] = dp[q] * a[q];
        }
        uint16_t* out = e.dgu + m * (2 * static_cast<int64_t>(e.f));
        *reinterpret_cast<u32x4*>(out + n) = pack8(dg);
        *reinterpret_cast<u32x4*>(out + e.f + n) = pack8(du);
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

// -------------------------------------------------------------- the kernel

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

template <Layout LA, Layout LB, EpiKind KIND, int PAIR, int WAVES>
__global__ void __launch_bounds__(WAVES * 64, 1) gemm_kernel(GemmParams p) {
  constexpr int NS = WAVES == 8 ? 2 : 4;     // 32-column blocks per wave (half of them low)
  constexpr int PER = 16 / WAVES;           // copies per operand per stage per wave
  __shared__ __attribute__((aligned(16))) uint8_t a0[TILE_BYTES], b0[TILE_BYTES], a1[TILE_BYTES], b1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t a2[TILE_BYTES], b2[TILE_BYTES], a3[TILE_BYTES], b3[TILE_BYTES];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.B.split_rows ? (p.B.split_rows + 127) / 128 : (p.N + BN - 1) / BN;
  const int pid = xcd_remap(blockIdx.x, gridDim.x);
  const int group = GROUP_M * tiles_n;
  const int first_m = (pid / group) * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int tm = first_m + (pid % group) % gm;
  const int tn = (pid % group) / gm;
  const int m0 = tm * BM, n0 = tn * BN;
  const int wm = WAVES == 8 ? (wave >> 2) : (wave >> 1);
  const int wn = WAVES == 8 ? (wave & 3) : (wave & 1);
  int ncol[NS];
#pragma unroll
  for (int j = 0; j < NS / 2; ++j) {
    ncol[j] = lo_col<WAVES, PAIR>(wn, j);
    ncol[j + NS / 2] = ncol[j] + PAIR;
  }

  f32x16 acc[4][NS];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NS; ++j) acc[i][j] = f32x16{};

  KcRows<WAVES> ra{}, rb{};
  if constexpr (LA == Layout::KC) ra = kc_rows<WAVES>(p.A, m0, tm, wave, lane);
  if constexpr (LB == Layout::KC) rb = kc_rows<WAVES>(p.B, n0, tn, wave, lane);

  auto issue = [&](int k0, uint8_t* la, uint8_t* lb) {
    if constexpr (LA == Layout::KC) copy_kc<WAVES>(la, p.A, ra, k0, p.K, wave, lane);
    else copy_mn<WAVES>(la, p.A, m0, k0, p.K, wave, lane);
    if constexpr (LB == Layout::KC) copy_kc<WAVES>(lb, p.B, rb, k0, p.K, wave, lane);
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
    compute(kt * BK, la, lb);
  };
  issue(0, a0, b0);
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
  __syncthreads();   // every wave is done reading the stages before they become staging space

  // Epilogue: each wave stages R rows x (NS*32) columns of fp32 at a time in
  // its own 16 KB of LDS (column halves swapped on rows with bit 2 set, so the
  // two half-waves write different banks) and hands out 8-column vectors of
  // its low blocks with their PAIR partners.  Accumulator register i of a
  // lane: row 8(i/4) + 4(lane/32) + i%4, column lane%32 of its 32x32 tile.
  constexpr int C = NS * 32, R = 4096 / C, PASSES = 128 / R, MS_PER = R / 32;
  const int sb = WAVES == 8 ? wave : 2 * wave;    // this wave's 16 KB staging buffer
  uint8_t* mine = sb == 0 ? a0 : sb == 1 ? b0 : sb == 2 ? a1 : sb == 3 ? b1 : sb == 4 ? a2 : sb == 5 ? b2
                : sb == 6 ? a3 : b3;
  float* st = reinterpret_cast<float*>(mine);
#pragma unroll
  for (int pass = 0; pass < PASSES; ++pass) {
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
    constexpr int VEC = R * (NS / 2) * 4;  // 8-column vectors of the low blocks per pass
#pragma unroll 1
    for (int it = 0; it < VEC / 64; ++it) {
      const int idx = it * 64 + lane;
      const int rr = idx / ((NS / 2) * 4), v = idx % ((NS / 2) * 4);
      const int j = v >> 2, c8 = (v & 3) * 8;
      const int flip = ((rr >> 2) & 1) << 4;
      const float4* lo4 = reinterpret_cast<const float4*>(st + rr * C + ((j * 32 + c8) ^ flip));
      const float4* hi4 = reinterpret_cast<const float4*>(st + rr * C + (((j + NS / 2) * 32 + c8) ^ flip));
      const float4 l0 = lo4[0], l1 = lo4[1], h0 = hi4[0], h1 = hi4[1];
      float lo[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
      float hi[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
      const int64_t m = static_cast<int64_t>(m0) + wm * 128 + pass * R + rr;
      epilogue<KIND, PAIR>(p, m, tn, ncol[j] + c8, lo, hi);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
  }
  (void)n0;
}

int gemm_waves() {
  static int w = [] {
    const char* e = getenv("L4D_GEMM_WAVES");
    return (e && atoi(e) == 4) ? 4 : 8;
  }();
  return w;
}

template <Layout LA, Layout LB, EpiKind KIND, int PAIR>
hipError_t launch(const GemmParams& p, hipStream_t stream) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.B.split_rows ? (p.B.split_rows + 127) / 128 : (p.N + BN - 1) / BN;
  if (gemm_waves() == 4)
    hipLaunchKernelGGL((gemm_kernel<LA, LB, KIND, PAIR, 4>), dim3(tiles_m * tiles_n), dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL((gemm_kernel<LA, LB, KIND, PAIR, 8>), dim3(tiles_m * tiles_n), dim3(512), 0, stream, p);
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
  } else if (la == L::KC && lb == L::MN) {
    if (k == E::SwiGLUBwd) return launch<L::KC, L::MN, E::SwiGLUBwd, 128>(p, stream);
    if (k == E::ResidualSP) return launch<L::KC, L::MN, E::ResidualSP, 128>(p, stream);
    if (k == E::StoreBF16) return launch<L::KC, L::MN, E::StoreBF16, 128>(p, stream);
  } else if (la == L::MN && lb == L::MN) {
    if (k == E::AccF32) return launch<L::MN, L::MN, E::AccF32, 128>(p, stream);
  }
  return hipErrorInvalidValue;     // a layout / epilogue pairing the layer never uses
}

}  // namespace l4d
