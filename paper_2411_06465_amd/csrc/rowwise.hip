// Memory-bound row kernels: RMSNorm forward/backward, the gain-gradient
// reduction, the RoPE angle table, the vocabulary-parallel cross-entropy (bf16
// logits, or FP32 logits kept as the softmax) and the vocabulary-parallel
// embedding lookup and its gradient.
// One wave (64 lanes) owns one row; every global access is a 16-byte vector.
#include <math.h>

#include "kernels.h"

namespace l4d {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ void unpack8(u32x4 u, float* v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(u[i] << 16);
    v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ u32x4 pack8(const float* v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{v[2 * i], v[2 * i + 1]}, bf16x2));
  return r;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

constexpr int kMaxChunks = 16;   // h <= 64 lanes * 16 chunks * 8 = 8192

// ------------------------------------------------------------------ RMSNorm

// One wave per row.  All of the row's loads are issued before the first use,
// so that a wave keeps its whole row (8 KB at h = 4096) in flight: a use right
// after each load waits for it and leaves one kilobyte in flight per wave.
// CPT > 0: h = 512 CPT (every lane holds CPT chunks, no bounds); CPT = 0: any
// h that is a multiple of 8.
template <int CPT>
__global__ void __launch_bounds__(256) rmsnorm_fwd_kernel(const uint16_t* __restrict__ x,
                                                          const uint16_t* __restrict__ gain,
                                                          uint16_t* __restrict__ y, uint16_t* __restrict__ x_copy,
                                                          int64_t rows, int32_t h, float eps) {
  constexpr int NC = CPT > 0 ? CPT : kMaxChunks;
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int nch = CPT > 0 ? 64 * CPT : h / 8;
  const u32x4* xr = reinterpret_cast<const u32x4*>(x + row * h);
  const u32x4* gr = reinterpret_cast<const u32x4*>(gain);
  u32x4 v[NC], gv[NC];
#pragma unroll
  for (int it = 0; it < NC; ++it) {
    const int c = lane + 64 * it;
    if (CPT > 0 || c < nch) v[it] = __builtin_nontemporal_load(&xr[c]);     // read once
  }
  // the gain too, before any store: a load issued after a store waits for it
#pragma unroll
  for (int it = 0; it < NC; ++it) {
    const int c = lane + 64 * it;
    if (CPT > 0 || c < nch) gv[it] = gr[c];
  }
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < NC; ++it) {
    const int c = lane + 64 * it;
    if (CPT > 0 || c < nch) {
      float f[8];
      unpack8(v[it], f);
#pragma unroll
      for (int j = 0; j < 8; ++j) ss += f[j] * f[j];
    }
  }
  if (x_copy) {     // the input, kept for the backward
    u32x4* cr = reinterpret_cast<u32x4*>(x_copy + row * h);
#pragma unroll
    for (int it = 0; it < NC; ++it) {
      const int c = lane + 64 * it;
      if (CPT > 0 || c < nch) cr[c] = v[it];
    }
  }
  const float rstd = rsqrtf(wave_sum(ss) / h + eps);
  u32x4* yr = reinterpret_cast<u32x4*>(y + row * h);
#pragma unroll
  for (int it = 0; it < NC; ++it) {
    const int c = lane + 64 * it;
    if (CPT > 0 || c < nch) {
      float f[8], g[8];
      unpack8(v[it], f);
      unpack8(gv[it], g);
#pragma unroll
      for (int j = 0; j < 8; ++j) f[j] = f[j] * rstd * g[j];
      yr[c] = pack8(f);
    }
  }
}

// Eight consecutive values of a bf16 row (one 16-byte load) or an fp32 row (two).
template <bool F32>
struct Vec8 {
  u32x4 v;
};
typedef float f32x4 __attribute__((ext_vector_type(4)));
template <>
struct Vec8<true> {
  f32x4 a, b;
};
template <bool F32>
__device__ __forceinline__ Vec8<F32> load8(const void* row, int c) {      // read-once rows: non-temporal
  if constexpr (F32) {
    const f32x4* p = reinterpret_cast<const f32x4*>(row) + 2 * c;
    return Vec8<true>{__builtin_nontemporal_load(p), __builtin_nontemporal_load(p + 1)};
  } else {
    return Vec8<false>{__builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row) + c)};
  }
}
template <bool F32>
__device__ __forceinline__ void unpack(const Vec8<F32>& u, float* v) {
  if constexpr (F32) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[i] = u.a[i];
      v[4 + i] = u.b[i];
    }
  } else {
    unpack8(u.v, v);
  }
}

// Grid-stride over rows, one 256-thread block per row: thread t owns the
// 8-column chunks t + 256 it (it < CPT, h <= 2048 * CPT) of every row, so it
// keeps its columns' partial sums of dy*xhat in registers and writes them to
// partial[blockIdx.x][h] at the end.  The two row sums go through LDS,
// double-buffered by row parity so one barrier per row suffices.
// DY32: the incoming gradient d(out) is fp32 (else bf16); RES: the residual
// gradient added to the result is absent (0), bf16 (1) or fp32 (2); OUT32:
// the result is also stored in fp32.
template <int CPT, bool DY32, int RES, bool OUT32>
__global__ void __launch_bounds__(256) rmsnorm_bwd_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ gain, const void* __restrict__ dy,
    const void* __restrict__ dres, uint16_t* __restrict__ dx, float* __restrict__ dx32, float* __restrict__ partial,
    int64_t rows, int32_t h, float eps) {
  constexpr bool R32 = RES == 2;
  __shared__ float sums[2][4][2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nch = h / 8;
  float acc[CPT][8];
#pragma unroll
  for (int it = 0; it < CPT; ++it)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[it][j] = 0.f;
  const u32x4* gr = reinterpret_cast<const u32x4*>(gain);
  u32x4 gv[CPT];
  const int64_t dsz = DY32 ? 4 : 2, rsz = R32 ? 4 : 2;
  // row `row`'s x, d(out) and residual gradient into (a, b, r); every lane
  // loads (a lane past the row end reloads the row's last chunk, unused), so
  // the number of loads in flight is fixed and the waits for a row count exactly
  auto load_row = [&](int64_t row, u32x4 (&a)[CPT], Vec8<DY32> (&b)[CPT], Vec8<R32> (&r)[CPT])
                      __attribute__((always_inline)) {
    const u32x4* xr = reinterpret_cast<const u32x4*>(x + row * h);
    const void* dr = static_cast<const uint8_t*>(dy) + row * h * dsz;
    const void* rr = RES ? static_cast<const uint8_t*>(dres) + row * h * rsz : nullptr;
#pragma unroll
    for (int it = 0; it < CPT; ++it) {
      const int c = min(tid + 256 * it, nch - 1);
      a[it] = __builtin_nontemporal_load(&xr[c]);
      b[it] = load8<DY32>(dr, c);
      if constexpr (RES != 0) r[it] = load8<R32>(rr, c);
    }
  };
#pragma unroll
  for (int it = 0; it < CPT; ++it) gv[it] = gr[min(tid + 256 * it, nch - 1)];
  int parity = 0;
  // one row: the two row sums, then dx and the gain partials.  A lane past the
  // row end holds a copy of the last chunk (loads clamped), so it stores the
  // same values to the same place as the chunk's own lane, and no store is
  // conditional; it leaves the row sums and the gain partials alone.
  auto process = [&](int64_t row, const u32x4 (&xv)[CPT], const Vec8<DY32> (&dv)[CPT], const Vec8<R32> (&rv)[CPT])
                     __attribute__((always_inline)) {
    float ss = 0.f, dot = 0.f;
#pragma unroll
    for (int it = 0; it < CPT; ++it) {
      const int c = tid + 256 * it;
      if (c < nch) {
        float f[8], d[8], g[8];
        unpack8(xv[it], f);
        unpack<DY32>(dv[it], d);
        unpack8(gv[it], g);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          ss += f[j] * f[j];
          dot += g[j] * d[j] * f[j];
        }
      }
    }
    ss = wave_sum(ss);
    dot = wave_sum(dot);
    if (lane == 0) {
      sums[parity][wave][0] = ss;
      sums[parity][wave][1] = dot;
    }
    __syncthreads();
    ss = (sums[parity][0][0] + sums[parity][1][0]) + (sums[parity][2][0] + sums[parity][3][0]);
    dot = (sums[parity][0][1] + sums[parity][1][1]) + (sums[parity][2][1] + sums[parity][3][1]);
    parity ^= 1;
    const float rstd = rsqrtf(ss / h + eps);
    const float c_mean = dot * rstd / h;        // mean over the row of (gain*dy) * xhat
    u32x4* out = reinterpret_cast<u32x4*>(dx + row * h);
    float4* out32 = OUT32 ? reinterpret_cast<float4*>(dx32 + row * h) : nullptr;
#pragma unroll
    for (int it = 0; it < CPT; ++it) {
      const int c = min(tid + 256 * it, nch - 1);
      const float own = tid + 256 * it < nch ? 1.f : 0.f;
      float f[8], d[8], g[8], r[8];
      unpack8(xv[it], f);
      unpack<DY32>(dv[it], d);
      unpack8(gv[it], g);
      if constexpr (RES != 0) {
        unpack<R32>(rv[it], r);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) r[j] = 0.f;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float xh = f[j] * rstd;
        acc[it][j] += own * (d[j] * xh);
        r[j] += rstd * (g[j] * d[j] - xh * c_mean);
      }
      out[c] = pack8(r);
      if constexpr (OUT32) {
        out32[2 * c] = make_float4(r[0], r[1], r[2], r[3]);
        out32[2 * c + 1] = make_float4(r[4], r[5], r[6], r[7]);
      }
    }
  };
  const int64_t G = gridDim.x, last = rows - 1;
  if constexpr (CPT <= 2 && DY32 && RES == 2) {
    // The read-heaviest form (10 of its 12 bytes per element are reads) keeps
    // two rows in flight, in three register sets: rows row + G and row + 2G
    // load while row is processed (a load past the last row reloads the last
    // row, unused).  On 268 MB cache-cold tensors: 302 -> 287 us; the lighter
    // forms measured no better.
    u32x4 xa[CPT], xb[CPT], xc[CPT];
    Vec8<DY32> da[CPT], db[CPT], dc[CPT];
    Vec8<R32> ra[CPT], rb[CPT], rc[CPT];
    int64_t row = blockIdx.x;
    if (row < rows) {
      load_row(row, xa, da, ra);
      load_row(min(row + G, last), xb, db, rb);
    }
    for (; row < rows; row += 3 * G) {
      load_row(min(row + 2 * G, last), xc, dc, rc);
      process(row, xa, da, ra);
      if (row + G >= rows) break;
      load_row(min(row + 3 * G, last), xa, da, ra);
      process(row + G, xb, db, rb);
      if (row + 2 * G >= rows) break;
      load_row(min(row + 4 * G, last), xb, db, rb);
      process(row + 2 * G, xc, dc, rc);
    }
  } else {
    u32x4 xv[CPT], xn[CPT];
    Vec8<DY32> dv[CPT], dn[CPT];
    Vec8<R32> rv[CPT], rn[CPT];
    if (static_cast<int64_t>(blockIdx.x) < rows) load_row(blockIdx.x, xn, dn, rn);
    for (int64_t row = blockIdx.x; row < rows; row += G) {
#pragma unroll
      for (int it = 0; it < CPT; ++it) {
        xv[it] = xn[it];
        dv[it] = dn[it];
        if constexpr (RES != 0) rv[it] = rn[it];
      }
      // the next row's loads fly under this row's reductions and stores
      if (row + G < rows) load_row(row + G, xn, dn, rn);
      process(row, xv, dv, rv);
    }
  }
  float* pr = partial + static_cast<int64_t>(blockIdx.x) * h;
#pragma unroll
  for (int it = 0; it < CPT; ++it) {
    const int c = tid + 256 * it;
    if (c < nch) {
      reinterpret_cast<float4*>(pr + c * 8)[0] = make_float4(acc[it][0], acc[it][1], acc[it][2], acc[it][3]);
      reinterpret_cast<float4*>(pr + c * 8)[1] = make_float4(acc[it][4], acc[it][5], acc[it][6], acc[it][7]);
    }
  }
}

// Column sums of partial[n][h] in two deterministic levels (no atomics):
// level 1 sums each slice of 64 rows into the slice's first row, in place,
// a block per (64 columns, slice) with its 4 waves taking every 4th row;
// level 2 adds the slice sums, in slice order, into out.
__global__ void __launch_bounds__(256) reduce_slices_kernel(float* __restrict__ partial, int32_t n, int32_t h) {
  __shared__ float s4[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lane;
  const int r0 = blockIdx.y * 64, r1 = min(r0 + 64, n);
  float s = 0.f;
  if (col < h) {
    int i = r0 + wave;
    for (; i + 12 < r1; i += 16) {     // four independent loads in flight
      const float a = partial[static_cast<int64_t>(i) * h + col];
      const float b = partial[static_cast<int64_t>(i + 4) * h + col];
      const float c = partial[static_cast<int64_t>(i + 8) * h + col];
      const float d = partial[static_cast<int64_t>(i + 12) * h + col];
      s += (a + b) + (c + d);
    }
    for (; i < r1; i += 4) s += partial[static_cast<int64_t>(i) * h + col];
  }
  s4[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && col < h)
    partial[static_cast<int64_t>(r0) * h + col] = (s4[0][lane] + s4[1][lane]) + (s4[2][lane] + s4[3][lane]);
}

// One level for at most 256 partial rows: a block per 64 columns, its 4 waves
// taking every 4th row (four loads in flight each), then out += the column sums.
__global__ void __launch_bounds__(256) reduce_all_kernel(const float* __restrict__ partial, int32_t n, int32_t h,
                                                        float* __restrict__ out) {
  __shared__ float s4[4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (col < h) {
    int i = wave;
    for (; i + 12 < n; i += 16) {
      const float a = partial[static_cast<int64_t>(i) * h + col];
      const float b = partial[static_cast<int64_t>(i + 4) * h + col];
      const float c = partial[static_cast<int64_t>(i + 8) * h + col];
      const float d = partial[static_cast<int64_t>(i + 12) * h + col];
      s += (a + b) + (c + d);
    }
    for (; i < n; i += 4) s += partial[static_cast<int64_t>(i) * h + col];
  }
  s4[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && col < h) out[col] += (s4[0][lane] + s4[1][lane]) + (s4[2][lane] + s4[3][lane]);
}

__global__ void __launch_bounds__(256) add_slices_kernel(const float* __restrict__ partial, int32_t n_slices,
                                                         int32_t h, float* __restrict__ out) {
  const int col = blockIdx.x * 256 + threadIdx.x;
  if (col >= h) return;
  float s = 0.f;
  for (int i = 0; i < n_slices; ++i) s += partial[static_cast<int64_t>(i) * 64 * h + col];
  out[col] += s;
}

// ------------------------------------------------------------------ RoPE table

__global__ void rope_table_kernel(float2* tab, ChunkMap map, int32_t rows, int32_t d_h, double log_base) {
  const int half = d_h / 2;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= static_cast<int64_t>(rows) * half) return;
  const int i = static_cast<int>(idx / half), j = static_cast<int>(idx % half);
  const int ci = i / map.chunk_len;
  const int64_t pos = static_cast<int64_t>(map.chunk_id[ci]) * map.chunk_len + (i - ci * map.chunk_len);
  const double ang = static_cast<double>(pos) * exp(-2.0 * j / d_h * log_base);
  double s, c;
  sincos(ang, &s, &c);
  tab[idx] = make_float2(static_cast<float>(c), static_cast<float>(s));
}

// ------------------------------------------------------------------ cross-entropy
// One 256-thread block per token row of bf16 logits [n][v_t] (v_t % 8 == 0).
// logits and dlogits may be the same buffer (the LM head overwrites the logits
// with their gradient in place), so neither is declared __restrict__.

__global__ void __launch_bounds__(256) xent_rows_kernel(
    const uint16_t* logits, int32_t v_t, int64_t v0, const int64_t* __restrict__ targets,
    const float* __restrict__ peer_lse, const float* __restrict__ peer_z, float grad_scale,
    float* __restrict__ loss, uint16_t* dlogits) {
  __shared__ float red_m[4], red_s[4];
  __shared__ float bcast;
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const u32x4* lr = reinterpret_cast<const u32x4*>(logits + row * v_t);
  const int nch = v_t / 8;
  // one read of the row: running maximum and the sum of exponentials relative to it
  float mx = -INFINITY, se = 0.f;
  for (int c = threadIdx.x; c < nch; c += 256) {
    float f[8];
    unpack8(lr[c], f);
    float m8 = f[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) m8 = fmaxf(m8, f[j]);
    if (m8 > mx) {
      se *= __expf(mx - m8);       // 0 while mx is -inf
      mx = m8;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) se += __expf(f[j] - mx);
  }
  // combine (max, sum) pairs across the wave, then the four waves
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(mx, o, 64), s2 = __shfl_xor(se, o, 64);
    const float m = fmaxf(mx, m2);
    se = (mx == -INFINITY ? 0.f : se * __expf(mx - m)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - m));
    mx = m;
  }
  if (lane == 0) {
    red_m[wave] = mx;
    red_s[wave] = se;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) sum += red_m[w] == -INFINITY ? 0.f : red_s[w] * __expf(red_m[w] - m);
    float lse = m + logf(sum);
    if (peer_lse) {
      const float p = peer_lse[row];
      const float hi = fmaxf(lse, p), lo = fminf(lse, p);
      lse = hi + log1pf(__expf(lo - hi));
    }
    const int64_t tgt = targets[row] - v0;
    float z;
    if (tgt >= 0 && tgt < v_t) z = __uint_as_float(static_cast<uint32_t>(logits[row * v_t + tgt]) << 16);
    else z = peer_z ? peer_z[row] : 0.f;
    loss[row] = lse - z;
    bcast = lse;
  }
  __syncthreads();
  const float lse = bcast;
  const int64_t tgt = targets[row] - v0;
  u32x4* dr = reinterpret_cast<u32x4*>(dlogits + row * v_t);
  for (int c = threadIdx.x; c < nch; c += 256) {
    float f[8];
    unpack8(lr[c], f);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float g = __expf(f[j] - lse);
      if (c * 8 + j == tgt) g -= 1.0f;
      f[j] = g * grad_scale;
    }
    dr[c] = pack8(f);
  }
}


// FP32 logits [n][v_t] (v_t % 4 == 0), one 256-thread block per row: the loss,
// and the row overwritten with the softmax exp(z - LSE) over the whole
// vocabulary (LSE combined with the other shards' log-sum-exp).
__global__ void __launch_bounds__(256) xent_probs_kernel(
    float* __restrict__ lp, int32_t v_t, int64_t v0, const int64_t* __restrict__ targets,
    const float* __restrict__ peer_lse, const float* __restrict__ peer_z, float* __restrict__ loss) {
  __shared__ float red_m[4], red_s[4];
  __shared__ float bcast;
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float4* r4 = reinterpret_cast<float4*>(lp + row * v_t);
  const int nch = v_t / 4;
  // one pass: running maximum and the sum of exponentials relative to it
  float mx = -INFINITY, se = 0.f;
  for (int c = threadIdx.x; c < nch; c += 256) {
    const float4 f = r4[c];
    const float m4 = fmaxf(fmaxf(f.x, f.y), fmaxf(f.z, f.w));
    if (m4 > mx) {
      se *= __expf(mx - m4);       // 0 while mx is -inf
      mx = m4;
    }
    se += __expf(f.x - mx) + __expf(f.y - mx) + __expf(f.z - mx) + __expf(f.w - mx);
  }
  // combine (max, sum) pairs across the wave, then the four waves
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(mx, o, 64), s2 = __shfl_xor(se, o, 64);
    const float m = fmaxf(mx, m2);
    se = (mx == -INFINITY ? 0.f : se * __expf(mx - m)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - m));
    mx = m;
  }
  if (lane == 0) {
    red_m[wave] = mx;
    red_s[wave] = se;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) sum += red_m[w] == -INFINITY ? 0.f : red_s[w] * __expf(red_m[w] - m);
    float lse = m + logf(sum);
    if (peer_lse) {
      const float p = peer_lse[row];
      const float hi = fmaxf(lse, p), lo = fminf(lse, p);
      lse = hi + log1pf(__expf(lo - hi));
    }
    const int64_t tgt = targets[row] - v0;
    float z;
    if (tgt >= 0 && tgt < v_t) z = lp[row * v_t + tgt];
    else z = peer_z ? peer_z[row] : 0.f;
    loss[row] = lse - z;
    bcast = lse;
  }
  __syncthreads();
  const float lse = bcast;
  for (int c = threadIdx.x; c < nch; c += 256) {
    const float4 f = r4[c];
    r4[c] = make_float4(__expf(f.x - lse), __expf(f.y - lse), __expf(f.z - lse), __expf(f.w - lse));
  }
}

// dlogits = (softmax - onehot(target)) * grad_scale as bf16, 8 elements per
// thread over the flattened [n][v_t] (v_t % 8 == 0).
__global__ void __launch_bounds__(256) xent_grad_kernel(const float* __restrict__ probs, int64_t n8, int32_t v8,
                                                       int64_t v0, const int64_t* __restrict__ targets,
                                                       float grad_scale, uint16_t* __restrict__ dl) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n8) return;
  const int64_t row = i / v8;
  const int32_t col0 = static_cast<int32_t>(i - row * v8) * 8;
  const int64_t tgt = targets[row] - v0 - col0;
  const float4* p4 = reinterpret_cast<const float4*>(probs) + 2 * i;
  const float4 a = p4[0], b = p4[1];
  float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int j = 0; j < 8; ++j) f[j] = (j == tgt ? f[j] - 1.0f : f[j]) * grad_scale;
  reinterpret_cast<u32x4*>(dl)[i] = pack8(f);
}

// ------------------------------------------------------------------ embedding
// Rows of the gathered [b][s_c] token view are split between this rank's own
// sequence-parallel rows and the peers' rows as in the layer (SpRows below).

struct SpRows {
  int32_t s_c, s_sp, r, t;
  // logical row m -> (own row index) or (peer row index) | 0x80000000
  __device__ uint32_t map(int64_t m64) const {
    const int32_t m = static_cast<int32_t>(m64);
    if (t == 1) return static_cast<uint32_t>(m);
    const int32_t bi = m / s_c, i = m - bi * s_c, lo = r * s_sp;
    if (i >= lo && i < lo + s_sp) return static_cast<uint32_t>(bi * s_sp + (i - lo));
    return static_cast<uint32_t>(bi * (t - 1) * s_sp + (i < lo ? i : i - s_sp)) | 0x80000000u;
  }
};

// One wave per gathered row: the table row when the id is in [v0, v0 + v_t),
// zeros otherwise.  Own rows: bf16(partial + receipt); peer rows: the partial.
__global__ void __launch_bounds__(256) embed_fwd_kernel(const int64_t* __restrict__ ids,
                                                       const uint16_t* __restrict__ w, int64_t v0, int32_t v_t,
                                                       int32_t h, int64_t rows, SpRows sp,
                                                       const uint16_t* __restrict__ receipt,
                                                       uint16_t* __restrict__ own, uint16_t* __restrict__ send) {
  const int lane = threadIdx.x & 63;
  const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (m >= rows) return;
  const int64_t j = ids[m] - v0;
  const bool hit = j >= 0 && j < v_t;
  const uint32_t o = sp.map(m);
  const bool mine = !(o & 0x80000000u);
  const int64_t orow = o & 0x7fffffffu;
  u32x4* dst = reinterpret_cast<u32x4*>((mine ? own : send) + orow * h);
  const u32x4* src = reinterpret_cast<const u32x4*>(w + (hit ? j : 0) * h);
  const u32x4* rc = (mine && receipt) ? reinterpret_cast<const u32x4*>(receipt + orow * h) : nullptr;
  for (int c = lane; c < h / 8; c += 64) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    const u32x4 v = hit ? src[c] : z;
    if (rc) {
      float a[8], b[8];
      unpack8(v, a);
      unpack8(rc[c], b);
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] += b[e];
      dst[c] = pack8(a);
    } else {
      dst[c] = v;
    }
  }
}

// One wave per gathered row of an fp32 sum: own rows -> bf16(sum + receipt),
// the peers' rows -> bf16(sum) into send (the residual epilogue of a GEMM
// whose K was summed in two parts).
__global__ void __launch_bounds__(256) sp_finish_kernel(const float* __restrict__ sum, int32_t h, int64_t rows,
                                                       SpRows sp, const uint16_t* __restrict__ receipt,
                                                       uint16_t* __restrict__ own, uint16_t* __restrict__ send) {
  const int lane = threadIdx.x & 63;
  const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (m >= rows) return;
  const uint32_t o = sp.map(m);
  const bool mine = !(o & 0x80000000u);
  const int64_t orow = o & 0x7fffffffu;
  const float4* src = reinterpret_cast<const float4*>(sum + m * h);
  u32x4* dst = reinterpret_cast<u32x4*>((mine ? own : send) + orow * h);
  const u32x4* rc = (mine && receipt) ? reinterpret_cast<const u32x4*>(receipt + orow * h) : nullptr;
  for (int c = lane; c < h / 8; c += 64) {
    const float4 a = src[2 * c], b = src[2 * c + 1];
    float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    if (rc) {
      float r[8];
      unpack8(rc[c], r);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] += r[e];
    }
    dst[c] = pack8(f);
  }
}

// One wave per gathered row whose id is in range: dW[id - v0] += dY[row]
// (fp32 atomic adds: rows that share an id add in no fixed order).
__global__ void __launch_bounds__(256) embed_bwd_kernel(const int64_t* __restrict__ ids, RowSrc dy, int64_t v0,
                                                       int32_t v_t, int32_t h, int64_t rows, float* __restrict__ dw) {
  const int lane = threadIdx.x & 63;
  const int64_t m = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (m >= rows) return;
  const int64_t j = ids[m] - v0;
  if (j < 0 || j >= v_t) return;
  const u32x4* src = reinterpret_cast<const u32x4*>(dy.row(m));
  float* d = dw + j * h;
  for (int c = lane; c < h / 8; c += 64) {
    float f[8];
    unpack8(src[c], f);
#pragma unroll
    for (int e = 0; e < 8; ++e) unsafeAtomicAdd(d + c * 8 + e, f[e]);
  }
}

}  // namespace

hipError_t rmsnorm_fwd(const uint16_t* x, const uint16_t* gain, uint16_t* y, int64_t rows, int32_t h,
                       float eps, hipStream_t stream, uint16_t* x_copy) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((rows + 3) / 4));
  switch (h % 512 == 0 ? h / 512 : 0) {
    case 8: hipLaunchKernelGGL(rmsnorm_fwd_kernel<8>, grid, dim3(256), 0, stream, x, gain, y, x_copy, rows, h, eps); break;
    case 16: hipLaunchKernelGGL(rmsnorm_fwd_kernel<16>, grid, dim3(256), 0, stream, x, gain, y, x_copy, rows, h, eps); break;
    default: hipLaunchKernelGGL(rmsnorm_fwd_kernel<0>, grid, dim3(256), 0, stream, x, gain, y, x_copy, rows, h, eps);
  }
  return hipGetLastError();
}

int32_t rmsnorm_bwd_partials(int64_t rows) {
  return static_cast<int32_t>(rows < 256 ? rows : 256);     // one block per row, one per CU
}

hipError_t rmsnorm_bwd(const uint16_t* x, const uint16_t* gain, const NormBwdIo& io, float* partial,
                       int32_t n_partial, int64_t rows, int32_t h, float eps, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  const int cpl = (h + 2047) / 2048;
  const bool dy32 = io.dy_f32 != nullptr;
  const int res = io.dres_f32 ? 2 : io.dres ? 1 : 0;
  const bool out32 = io.dx_f32 != nullptr;
  const void* dy = dy32 ? static_cast<const void*>(io.dy_f32) : io.dy;
  const void* dres = res == 2 ? static_cast<const void*>(io.dres_f32) : io.dres;
  // the three forms the layer and the LM-head block use
#define L4D_RMS_BWD(C, D32, R, O32)                                                                            \
  hipLaunchKernelGGL((rmsnorm_bwd_kernel<C, D32, R, O32>), dim3(n_partial), dim3(256), 0, stream, x, gain, dy, \
                     dres, io.dx, io.dx_f32, partial, rows, h, eps)
#define L4D_RMS_BWD_FORM(C)                                                      \
  if (!dy32 && res == 0 && !out32) L4D_RMS_BWD(C, false, 0, false);              \
  else if (dy32 && res == 1 && out32) L4D_RMS_BWD(C, true, 1, true);             \
  else if (dy32 && res == 2 && !out32) L4D_RMS_BWD(C, true, 2, false);           \
  else return hipErrorInvalidValue;
  if (cpl <= 1) {
    L4D_RMS_BWD_FORM(1)
  } else if (cpl <= 2) {
    L4D_RMS_BWD_FORM(2)
  } else {
    L4D_RMS_BWD_FORM(4)
  }
#undef L4D_RMS_BWD_FORM
#undef L4D_RMS_BWD
  return hipGetLastError();
}

hipError_t reduce_rows_add(float* partial, int32_t n_partial, int32_t h, float* out, hipStream_t stream) {
  if (n_partial <= 0) return hipSuccess;
  if (n_partial <= 256) {
    hipLaunchKernelGGL(reduce_all_kernel, dim3((h + 63) / 64), dim3(256), 0, stream, partial, n_partial, h, out);
    return hipGetLastError();
  }
  const int slices = (n_partial + 63) / 64;
  hipLaunchKernelGGL(reduce_slices_kernel, dim3((h + 63) / 64, slices), dim3(256), 0, stream, partial, n_partial, h);
  hipLaunchKernelGGL(add_slices_kernel, dim3((h + 255) / 256), dim3(256), 0, stream, partial, slices, h, out);
  return hipGetLastError();
}

hipError_t rope_table(float2* tab, ChunkMap map, int32_t rows, int32_t d_h, float base, hipStream_t stream) {
  const int64_t n = static_cast<int64_t>(rows) * (d_h / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream,
                     tab, map, rows, d_h, log(static_cast<double>(base)));
  return hipGetLastError();
}

hipError_t xent_rows(const uint16_t* logits, int64_t n, int32_t v_t, int64_t v0, const int64_t* targets,
                     const float* peer_lse, const float* peer_z, float grad_scale, float* loss,
                     uint16_t* dlogits, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(xent_rows_kernel, dim3(static_cast<unsigned>(n)), dim3(256), 0, stream, logits, v_t, v0,
                     targets, peer_lse, peer_z, grad_scale, loss, dlogits);
  return hipGetLastError();
}

hipError_t xent_probs(float* logits, int64_t n, int32_t v_t, int64_t v0, const int64_t* targets,
                      const float* peer_lse, const float* peer_z, float* loss, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(xent_probs_kernel, dim3(static_cast<unsigned>(n)), dim3(256), 0, stream, logits, v_t, v0,
                     targets, peer_lse, peer_z, loss);
  return hipGetLastError();
}

hipError_t xent_grad(const float* probs, int64_t n, int32_t v_t, int64_t v0, const int64_t* targets,
                     float grad_scale, uint16_t* dlogits, hipStream_t stream) {
  const int64_t n8 = n * (v_t / 8);
  if (n8 <= 0) return hipSuccess;
  hipLaunchKernelGGL(xent_grad_kernel, dim3(static_cast<unsigned>((n8 + 255) / 256)), dim3(256), 0, stream, probs,
                     n8, v_t / 8, v0, targets, grad_scale, dlogits);
  return hipGetLastError();
}

hipError_t embed_fwd(const int64_t* ids, const uint16_t* w, int64_t v0, int32_t v_t, int32_t h, int64_t rows,
                     int32_t s_c, int32_t s_sp, int32_t r, int32_t t, const uint16_t* receipt, uint16_t* own,
                     uint16_t* send, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(embed_fwd_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream, ids, w,
                     v0, v_t, h, rows, SpRows{s_c, s_sp, r, t}, receipt, own, send);
  return hipGetLastError();
}

hipError_t sp_finish(const float* sum, int32_t h, int64_t rows, int32_t s_c, int32_t s_sp, int32_t r, int32_t t,
                     const uint16_t* receipt, uint16_t* own, uint16_t* send, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(sp_finish_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream, sum, h, rows,
                     SpRows{s_c, s_sp, r, t}, receipt, own, send);
  return hipGetLastError();
}

hipError_t embed_bwd(const int64_t* ids, RowSrc dy, int64_t v0, int32_t v_t, int32_t h, int64_t rows, float* dw,
                     hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(embed_bwd_kernel, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream, ids, dy,
                     v0, v_t, h, rows, dw);
  return hipGetLastError();
}

}  // namespace l4d
