// bf16 GEMM on the gfx950 matrix cores: C[m][n] = sum_k A(m,k) B(n,k), fp32
// accumulation, with the layer's fused epilogues.
//
// Tiling: one 512-thread workgroup (8 waves, 2 per SIMD) owns a 256x256 tile
// of C and walks K in steps of 64.  Both operand tiles (256 x 64 bf16 each)
// are double-buffered in LDS (128 KB); each wave computes a 128 x 64 block as
// 4 x 2 v_mfma_f32_32x32x16_bf16 accumulators.  Tiles are stored k-contiguous
// in LDS with an XOR swizzle of the 16-byte chunks so that 8 consecutive rows
// read by one MFMA fragment load hit distinct banks.  Operands whose
// reduction index is not contiguous in memory (the weight operand of dX, both
// operands of dW) are loaded as 8x8 blocks and transposed in registers on
// their way to LDS, so every fragment read is one 16-byte LDS load.
//
// The two 32-column accumulator blocks of a wave sit PAIR columns apart, so
// that one lane owns both members of a RoPE pair (i, i + d_h/2) or of a
// gate/up pair; the epilogue stages each wave's fp32 block through LDS and
// writes 8-column vectors.
#include "kernels.h"

namespace l4d {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 256, BN = 256, BK = 64, NT = 512;
constexpr int TILE_BYTES = 256 * BK * 2;            // one operand tile
constexpr int STAGE_LD = 68;                        // fp32 words per staged row
constexpr int STAGE_WAVE = 64 * STAGE_LD;           // fp32 words per wave
constexpr int LDS_BYTES = 8 * STAGE_WAVE * 4;       // 139264 >= 4 * TILE_BYTES
static_assert(LDS_BYTES >= 4 * TILE_BYTES, "LDS too small for the double buffer");
constexpr int GROUP_M = 8;

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 4);
}

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ float bf2f(uint32_t u16) { return __uint_as_float(u16 << 16); }

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

// Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous range of tiles so that neighbouring tiles share its L2.
__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
  const int X = 8;
  int per = nwg / X, rem = nwg % X, xcd = bid % X, local = bid / X;
  return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// -------------------------------------------------------------- operand movement
// Thread `tid` (0..255 of the half that loads this operand) moves one 8x8 block.

template <Layout L>
__device__ __forceinline__ void load_block(const Operand& op, int x0, int tile_idx, int k0, int K,
                                           int tid, u32x4 (&v)[8]) {
  const u32x4 zero = {0u, 0u, 0u, 0u};
  if constexpr (L == Layout::KC) {
    const int rb = tid >> 3, kb = tid & 7;
    const int k = k0 + kb * 8;
    const bool kok = k < K;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int xr = rb * 8 + j;
      int64_t gx;
      bool ok;
      if (op.split_rows) {
        const int i = tile_idx * 128 + (xr & 127);
        ok = i < op.split_rows;
        gx = (xr >= 128 ? op.split_off : 0) + i;
      } else {
        gx = x0 + xr;
        ok = gx < op.rows;
      }
      v[j] = (ok && kok) ? *reinterpret_cast<const u32x4*>(op.src.row(gx) + k) : zero;
    }
  } else {
    const int rb = tid & 31, kb = tid >> 5;
    const int x = x0 + rb * 8;
    const bool xok = x < op.rows;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = k0 + kb * 8 + j;
      v[j] = (xok && k < K) ? *reinterpret_cast<const u32x4*>(op.src.row(k) + x) : zero;
    }
  }
}

template <Layout L>
__device__ __forceinline__ void store_block(uint8_t* lds, int tid, const u32x4 (&v)[8]) {
  if constexpr (L == Layout::KC) {
    const int rb = tid >> 3, kb = tid & 7;
#pragma unroll
    for (int j = 0; j < 8; ++j) *reinterpret_cast<u32x4*>(lds + lds_off(rb * 8 + j, kb)) = v[j];
  } else {
    // v[j] holds k-row j of the block (8 consecutive x); emit x-row i (8 consecutive k).
    const int rb = tid & 31, kb = tid >> 5;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int d = i >> 1;
      u32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t a = v[2 * e][d], b = v[2 * e + 1][d];
        o[e] = (i & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
      }
      *reinterpret_cast<u32x4*>(lds + lds_off(rb * 8 + i, kb)) = o;
    }
  }
}

// -------------------------------------------------------------- epilogues

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

// lo: 8 columns starting at tile column `col`; hi: the 8 columns PAIR further.
template <int PAIR>
__device__ __forceinline__ void epilogue(const GemmParams& p, int64_t m, int tn, int col,
                                         float* lo, float* hi) {
  const EpiParams& e = p.epi;
  if (m >= p.M) return;
  const int n_lo = tn * BN + col;
  switch (e.kind) {
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

// -------------------------------------------------------------- the kernel

template <Layout LA, Layout LB, int PAIR>
__global__ void __launch_bounds__(NT) gemm_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];
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

  const int wm = wave >> 2, wn = wave & 3;
  constexpr int PW = PAIR / 32;
  const int c0 = (wn / PW) * (2 * PAIR) + (wn % PW) * 32;
  const int c1 = c0 + PAIR;

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  const bool loads_a = tid < 256;
  const int ltid = tid & 255;
  const int nk = (p.K + BK - 1) / BK;
  u32x4 stage[8];

  auto gload = [&](int kt) {
    if (loads_a) load_block<LA>(p.A, m0, tm, kt * BK, p.K, ltid, stage);
    else load_block<LB>(p.B, n0, tn, kt * BK, p.K, ltid, stage);
  };
  auto lstore = [&](int buf) {
    uint8_t* base = smem + buf * 2 * TILE_BYTES;
    if (loads_a) store_block<LA>(base, ltid, stage);
    else store_block<LB>(base + TILE_BYTES, ltid, stage);
  };

  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    const uint8_t* sa = smem + buf * 2 * TILE_BYTES;
    const uint8_t* sb = sa + TILE_BYTES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = kk * 2 + (lane >> 5);
      bf16x8 af[4], bf[2];
#pragma unroll
      for (int ms = 0; ms < 4; ++ms)
        af[ms] = *reinterpret_cast<const bf16x8*>(sa + lds_off(wm * 128 + ms * 32 + (lane & 31), ch));
      bf[0] = *reinterpret_cast<const bf16x8*>(sb + lds_off(c0 + (lane & 31), ch));
      bf[1] = *reinterpret_cast<const bf16x8*>(sb + lds_off(c1 + (lane & 31), ch));
#pragma unroll
      for (int ms = 0; ms < 4; ++ms)
#pragma unroll
        for (int ns = 0; ns < 2; ++ns)
          acc[ms][ns] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ms], bf[ns], acc[ms][ns], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: stage each wave's 128x64 block (two 64-row halves) as fp32 in
  // LDS, then hand out 8-column vectors.  MFMA 32x32 output layout: register i
  // of lane l is row 8*(i/4) + 4*(l/32) + i%4, column l%32.
  float* st = reinterpret_cast<float*>(smem) + wave * STAGE_WAVE;
#pragma unroll
  for (int ph = 0; ph < 2; ++ph) {
#pragma unroll
    for (int mm = 0; mm < 2; ++mm)
#pragma unroll
      for (int ns = 0; ns < 2; ++ns)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = mm * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
          st[r * STAGE_LD + ns * 32 + (lane & 31)] = acc[2 * ph + mm][ns][i];
        }
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int rr = pass * 16 + (lane >> 2);
      const int cc = (lane & 3) * 8;
      float lo[8], hi[8];
      const float* srow = st + rr * STAGE_LD + cc;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        lo[j] = srow[j];
        hi[j] = srow[32 + j];
      }
      const int64_t m = static_cast<int64_t>(m0) + wm * 128 + ph * 64 + rr;
      epilogue<PAIR>(p, m, tn, c0 + cc, lo, hi);
    }
    __syncthreads();
  }
  (void)n0;
}

template <Layout LA, Layout LB>
hipError_t launch(const GemmParams& p, int pair, hipStream_t stream) {
  const int tiles_m = (p.M + BM - 1) / BM;
  const int tiles_n = p.B.split_rows ? (p.B.split_rows + 127) / 128 : (p.N + BN - 1) / BN;
  const dim3 grid(tiles_m * tiles_n), block(NT);
  switch (pair) {
    case 32: hipLaunchKernelGGL((gemm_kernel<LA, LB, 32>), grid, block, 0, stream, p); break;
    case 64: hipLaunchKernelGGL((gemm_kernel<LA, LB, 64>), grid, block, 0, stream, p); break;
    default: hipLaunchKernelGGL((gemm_kernel<LA, LB, 128>), grid, block, 0, stream, p); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t gemm(const GemmParams& p, Layout la, Layout lb, hipStream_t stream) {
  if (p.M <= 0 || p.N <= 0 || p.K <= 0) return hipSuccess;
  int pair = 128;
  if (p.epi.kind == EpiKind::QkvRope) pair = p.epi.d_h / 2;
  if (la == Layout::KC && lb == Layout::KC) return launch<Layout::KC, Layout::KC>(p, pair, stream);
  if (la == Layout::KC && lb == Layout::MN) return launch<Layout::KC, Layout::MN>(p, pair, stream);
  if (la == Layout::MN && lb == Layout::MN) return launch<Layout::MN, Layout::MN>(p, pair, stream);
  return launch<Layout::MN, Layout::KC>(p, pair, stream);
}

}  // namespace l4d
