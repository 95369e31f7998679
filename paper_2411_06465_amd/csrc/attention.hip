// Causal grouped-query attention on the gfx950 matrix cores, FlashAttention
// style: the forward keeps only the output and the per-row log-sum-exp, the
// backward recomputes the probabilities from Q, K and the log-sum-exp
// (the activation accounting of Sec. 3.2 counts QK^T and softmax as zero).
//
// Keys come as up to kMaxSeg runs with consecutive global positions: the
// rank's own context-parallel chunks and the remote chunks of the other CP
// ranks.  A key is visible to a query iff key position <= query position.
//
// Layout choices (gfx950, wave64, v_mfma_f32_32x32x16_bf16):
//  * scores are computed transposed, S^T = K Q^T, so that each lane owns one
//    query column of the accumulator; row statistics are then per-lane
//    scalars plus one cross-half exchange, and the bf16 probabilities already
//    sit in the B-operand layout of the next product O^T += V^T P^T (the
//    contraction index is permuted consistently on both operands).
//  * V (and, in the backward, Q^T, dO^T, K^T) are transposed in registers on
//    their way into LDS; K-like tiles are stored d-contiguous with an XOR
//    swizzle of the 16-byte chunks, transposed tiles token-contiguous with an
//    XOR swizzle of the 8-byte units.
//  * dK/dV accumulate over all q-heads of a kv-head inside one workgroup, and
//    dQ has its own kernel, so there are no atomics and results are
//    deterministic.
#include <math.h>

#include "kernels.h"

namespace l4d {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}
__device__ __forceinline__ float lo16(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi16(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------ LDS tiles
// R tile: [rows][D] bf16, 16-byte chunk c of row r at ((c ^ (r & 7)) << 4).
template <int D>
__device__ __forceinline__ int r_off(int row, int chunk) {
  return row * (D * 2) + ((chunk ^ (row & 7)) << 4);
}
// T tile: [D][64] bf16 (64 tokens per d-row), 8-byte unit u of row d at ((u ^ (d & 15)) << 3).
__device__ __forceinline__ int t_off(int drow, int unit) { return drow * 128 + ((unit ^ (drow & 15)) << 3); }

// Write an 8 (tokens) x 8 (d) block, v[j] = token t0+j, d-chunk dc.
template <int D>
__device__ __forceinline__ void put_r(uint8_t* lds, int t0, int dc, const u32x4 (&v)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) *reinterpret_cast<u32x4*>(lds + r_off<D>(t0 + j, dc)) = v[j];
}
__device__ __forceinline__ void put_t(uint8_t* lds, int t0, int dc, const u32x4 (&v)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int d = i >> 1;
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t a = v[2 * e][d], b = v[2 * e + 1][d];
      o[e] = (i & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
    const int drow = dc * 8 + i;
    *reinterpret_cast<u32x2*>(lds + t_off(drow, t0 >> 2)) = u32x2{o[0], o[1]};
    *reinterpret_cast<u32x2*>(lds + t_off(drow, (t0 >> 2) + 1)) = u32x2{o[2], o[3]};
  }
}

// A-operand fragment from an R tile: rows base + lane%32, d-chunk 2*kk + lane/32.
template <int D>
__device__ __forceinline__ bf16x8 frag_r(const uint8_t* lds, int base, int kk, int lane) {
  return *reinterpret_cast<const bf16x8*>(lds + r_off<D>(base + (lane & 31), 2 * kk + (lane >> 5)));
}
// A-operand fragment from a T tile: d-row drow0 + lane%32; the 16 contraction
// slots of token group g16 (tokens 16*g16 .. +15) are ordered like the lanes'
// accumulator rows of a 32x32 MFMA: slots 0-3 -> tokens 4*hh+0..3,
// slots 4-7 -> tokens 8+4*hh+0..3, hh = lane/32.
__device__ __forceinline__ bf16x8 frag_t(const uint8_t* lds, int drow0, int g16, int lane) {
  const int drow = drow0 + (lane & 31);
  const int u = g16 * 4 + (lane >> 5);
  const u32x2 a = *reinterpret_cast<const u32x2*>(lds + t_off(drow, u));
  const u32x2 b = *reinterpret_cast<const u32x2*>(lds + t_off(drow, u + 2));
  return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
}
// B-operand fragment from 8 accumulator registers i0..i0+7 (probabilities).
__device__ __forceinline__ bf16x8 frag_acc(const f32x16& s, int i0) {
  return __builtin_bit_cast(bf16x8, u32x4{pack2(s[i0], s[i0 + 1]), pack2(s[i0 + 2], s[i0 + 3]),
                                          pack2(s[i0 + 4], s[i0 + 5]), pack2(s[i0 + 6], s[i0 + 7])});
}
// Row of accumulator register i for this lane (32x32 MFMA output layout).
__device__ __forceinline__ int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

__device__ __forceinline__ int qpos(const ChunkMap& m, int row) {
  const int c = row / m.chunk_len;
  return m.chunk_id[c] * m.chunk_len + (row - c * m.chunk_len);
}

// Locate key tile `tile` (of `tsz` tokens) across the segments.
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
__device__ __forceinline__ int total_tiles(const AttnParams& p, int tsz) {
  int acc = 0;
  for (int s = 0; s < p.n_seg; ++s) acc += (p.seg[s].n + tsz - 1) / tsz;
  return acc;
}

// Load an 8-token x 8-d block of K or V (or Q / dO) from global; rows past n are zero.
__device__ __forceinline__ void load8(const uint16_t* base, int64_t ld, int t0, int n, int dcol,
                                      u32x4 (&v)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
    v[j] = (t0 + j < n) ? *reinterpret_cast<const u32x4*>(base + static_cast<int64_t>(t0 + j) * ld + dcol)
                        : u32x4{0u, 0u, 0u, 0u};
}

// ------------------------------------------------------------------ forward
// grid: (q tiles of 128, a_t heads, b); block 256 = 4 waves x 32 queries.
template <int D>
__global__ void __launch_bounds__(256) attn_fwd_kernel(AttnParams p) {
  constexpr int KT = 64;                        // keys per tile
  constexpr int TILE = KT * D * 2;              // bytes of one K (R) or V^T (T) tile
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][2][TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_qt = (p.n_q + 127) / 128;
  const int qt = n_qt - 1 - blockIdx.x;         // heaviest tiles first
  const int hq = blockIdx.y, bi = blockIdx.z;
  const int hk = hq / (p.a_t / p.k_t);
  const int q_row0 = qt * 128;
  const int my_q = q_row0 + wave * 32 + (lane & 31);
  const bool q_ok = my_q < p.n_q;
  const int my_pos = q_ok ? qpos(p.qmap, my_q) : -1;
  const int blk_last = min(q_row0 + 127, p.n_q - 1);
  const int pos_min = qpos(p.qmap, q_row0), pos_max = qpos(p.qmap, blk_last);

  // Q fragments (B operand): query my_q, d-chunk 2kk + lane/32.
  bf16x8 qf[D / 16];
  {
    const uint16_t* qb = p.q + bi * p.q_bstride + static_cast<int64_t>(my_q) * p.q_ld + hq * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      qf[kk] = q_ok ? *reinterpret_cast<const bf16x8*>(qb + (2 * kk + (lane >> 5)) * 8) : bf16x8{};
  }

  const float c = p.scale * kLog2e;
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) o[i] = f32x16{};

  // The tiles this block must visit: visible to at least one of its queries.
  const int ntiles = total_tiles(p, KT);
  auto visible = [&](int tile, int& seg, int& t0) {
    if (!find_tile(p, tile, KT, seg, t0)) return false;
    return p.seg[seg].pos0 + t0 <= pos_max;
  };
  auto next_visible = [&](int from, int& seg, int& t0) {
    for (int t = from; t < ntiles; ++t)
      if (visible(t, seg, t0)) return t;
    return ntiles;
  };

  // Loader role: threads 0..127 move K blocks, 128..255 V blocks.
  const bool is_k = tid < 128;
  const int lt = tid & 127;
  const int tb = lt / (D / 8), dc = lt % (D / 8);     // token block (of 8), d-chunk
  const bool loader = tb < KT / 8;
  u32x4 stage[8];
  auto gload = [&](int seg, int t0) {
    if (!loader) return;
    const KvSeg& s = p.seg[seg];
    const uint16_t* base = (is_k ? s.k : s.v) + bi * s.bstride + hk * D;
    load8(base + static_cast<int64_t>(t0) * s.ld, s.ld, tb * 8, s.n - t0, dc * 8, stage);
  };
  auto lstore = [&](int buf) {
    if (!loader) return;
    if (is_k) put_r<D>(smem[buf][0], tb * 8, dc, stage);
    else put_t(smem[buf][1], tb * 8, dc, stage);
  };

  int seg, t0;
  int cur = next_visible(0, seg, t0);
  if (cur < ntiles) {
    gload(seg, t0);
    lstore(0);
  }
  __syncthreads();
  int buf = 0;
  while (cur < ntiles) {
    const int cseg = seg, ct0 = t0;
    const int nxt = next_visible(cur + 1, seg, t0);
    if (nxt < ntiles) gload(seg, t0);

    const KvSeg& s = p.seg[cseg];
    const int kpos0 = s.pos0 + ct0;
    const int kvalid = min(KT, s.n - ct0);
    const bool need_mask = (kpos0 + KT - 1 > pos_min) || (kvalid < KT);

    // S^T for 64 keys x 32 queries: two 32-key accumulators.
    f32x16 sc[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) sc[t2] = mfma(frag_r<D>(smem[buf][0], t2 * 32, kk, lane), qf[kk], sc[t2]);

    float mx = -INFINITY;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float v = sc[t2][i] * c;
        if (need_mask) {
          const int kr = t2 * 32 + acc_row(i, lane);
          if (kr >= kvalid || kpos0 + kr > my_pos) v = -INFINITY;
        }
        sc[t2][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float pr = exp2f(sc[t2][i] - m_use);
        sc[t2][i] = pr;
        rs += pr;
      }
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) o[dt] *= alpha;
    // O^T[d][q] += V^T[d][keys] P^T[keys][q]
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const bf16x8 pf = frag_acc(sc[t2], 8 * g);
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) o[dt] = mfma(frag_t(smem[buf][1], dt * 32, t2 * 2 + g, lane), pf, o[dt]);
      }

    if (nxt < ntiles) lstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!q_ok) return;
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;
  uint16_t* ob = p.o + bi * p.q_bstride + static_cast<int64_t>(my_q) * p.q_ld + hq * D;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + 4 * (lane >> 5);
      const u32x2 w = {pack2(o[dt][4 * jj] * inv, o[dt][4 * jj + 1] * inv),
                       pack2(o[dt][4 * jj + 2] * inv, o[dt][4 * jj + 3] * inv)};
      *reinterpret_cast<u32x2*>(ob + d) = w;
    }
  if (lane < 32)
    p.lse[(static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q + my_q] =
        (m_run + log2f(l_tot)) * kLn2;
}

// ------------------------------------------------------------------ backward: delta
// delta[b][h][q] = sum_d dO[q][h*D + d] * O[q][h*D + d]; one wave per (b, q) row.
template <int D>
__global__ void __launch_bounds__(256) attn_delta_kernel(AttnParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= static_cast<int64_t>(p.b) * p.n_q) return;
  const int64_t bi = row / p.n_q, q = row % p.n_q;
  const uint16_t* o = p.o + bi * p.q_bstride + q * p.q_ld;
  const uint16_t* d = p.dout + bi * p.q_bstride + q * p.q_ld;
  constexpr int CPH = D / 8;                 // 16-byte chunks per head
  const int nch = p.a_t * CPH;
  for (int c0 = 0; c0 < nch; c0 += 64) {
    const int c = c0 + lane;
    float s = 0.f;
    if (c < nch) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(o + c * 8);
      const u32x4 b = *reinterpret_cast<const u32x4*>(d + c * 8);
#pragma unroll
      for (int j = 0; j < 4; ++j) s += lo16(a[j]) * lo16(b[j]) + hi16(a[j]) * hi16(b[j]);
    }
#pragma unroll
    for (int off = CPH / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (c < nch && (c % CPH) == 0) {
      const int h = c / CPH;
      p.delta[(bi * p.a_t + h) * p.n_q + q] = s;
    }
  }
}

// ------------------------------------------------------------------ backward: dK, dV
// grid: (key blocks of 128 over all segments, k_t kv-heads, b); 4 waves x 32 keys.
// Loops over the a/k query heads of the kv-head and over 64-query tiles.
template <int D>
__global__ void __launch_bounds__(256) attn_bwd_dkdv_kernel(AttnParams p) {
  constexpr int QT = 64;
  constexpr int TILE = QT * D * 2;
  // [buf][Q, Q^T, dO, dO^T]
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][4][TILE];
  __shared__ float s_lse[2][QT], s_delta[2][QT];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hk = blockIdx.y, bi = blockIdx.z;
  const int group = p.a_t / p.k_t;
  int seg, k0;
  if (!find_tile(p, blockIdx.x, 128, seg, k0)) return;
  const KvSeg& S = p.seg[seg];
  const int kbase = k0 + wave * 32;               // this wave's first key (in the segment)
  const int my_key = kbase + (lane & 31);
  const bool key_ok = my_key < S.n;
  const int my_kpos = S.pos0 + my_key;
  const int blk_kpos0 = S.pos0 + k0;

  // K and V fragments (B operands), key my_key, d-chunk 2kk + lane/32.
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const int64_t off = bi * S.bstride + static_cast<int64_t>(my_key) * S.ld + hk * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const int dcol = (2 * kk + (lane >> 5)) * 8;
      kf[kk] = key_ok ? *reinterpret_cast<const bf16x8*>(S.k + off + dcol) : bf16x8{};
      vf[kk] = key_ok ? *reinterpret_cast<const bf16x8*>(S.v + off + dcol) : bf16x8{};
    }
  }
  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
    dk[i] = f32x16{};
    dv[i] = f32x16{};
  }
  const float c = p.scale * kLog2e;
  const int n_qt = (p.n_q + QT - 1) / QT;
  const int total = group * n_qt;
  // a query tile matters if its last query can see the block's first key
  auto wanted = [&](int it) {
    const int qt = it % n_qt;
    const int last = min(qt * QT + QT - 1, p.n_q - 1);
    return qpos(p.qmap, last) >= blk_kpos0;
  };
  auto next_wanted = [&](int from) {
    for (int it = from; it < total; ++it)
      if (wanted(it)) return it;
    return total;
  };
  // loaders: threads 0..127 Q blocks, 128..255 dO blocks (64 tokens x D)
  const bool is_q = tid < 128;
  const int lt = tid & 127;
  const int tb = lt / (D / 8), dc = lt % (D / 8);
  const bool loader = tb < QT / 8;
  u32x4 stage[8];
  auto gload = [&](int it) {
    const int hq = hk * group + it / n_qt, qt = it % n_qt;
    if (loader) {
      const uint16_t* base = (is_q ? p.q : p.dout) + bi * p.q_bstride + hq * D +
                             static_cast<int64_t>(qt * QT) * p.q_ld;
      load8(base, p.q_ld, tb * 8, p.n_q - qt * QT, dc * 8, stage);
    }
  };
  auto lstore = [&](int buf, int it) {
    const int hq = hk * group + it / n_qt, qt = it % n_qt;
    if (loader) {
      put_r<D>(smem[buf][is_q ? 0 : 2], tb * 8, dc, stage);
      put_t(smem[buf][is_q ? 1 : 3], tb * 8, dc, stage);
    }
    if (tid < QT) {
      const int q = qt * QT + tid;
      const int64_t idx = (static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q + q;
      s_lse[buf][tid] = q < p.n_q ? p.lse[idx] * kLog2e : INFINITY;
      s_delta[buf][tid] = q < p.n_q ? p.delta[idx] : 0.f;
    }
  };

  int cur = next_wanted(0);
  if (cur < total) {
    gload(cur);
    lstore(0, cur);
  }
  __syncthreads();
  int buf = 0;
  while (cur < total) {
    const int nxt = next_wanted(cur + 1);
    if (nxt < total) gload(nxt);
    const int qt = cur % n_qt;
    const int qr0 = qt * QT;
    const uint8_t* tq = smem[buf][0];
    const uint8_t* tqt = smem[buf][1];
    const uint8_t* tdo = smem[buf][2];
    const uint8_t* tdot = smem[buf][3];

    // S[q][key] and dP[q][key] for 64 queries (two 32-row halves) x 32 keys.
    f32x16 sc[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        sc[h2] = mfma(frag_r<D>(tq, h2 * 32, kk, lane), kf[kk], sc[h2]);
        dp[h2] = mfma(frag_r<D>(tdo, h2 * 32, kk, lane), vf[kk], dp[h2]);
      }
    // P = exp(S*scale - lse), dS = P (dP - delta), masked where key > query.
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int qr = h2 * 32 + acc_row(i, lane);
        const int q = qr0 + qr;
        float pr = 0.f;
        if (key_ok && q < p.n_q && my_kpos <= qpos(p.qmap, q)) pr = exp2f(sc[h2][i] * c - s_lse[buf][qr]);
        sc[h2][i] = pr;
        dp[h2][i] = pr * (dp[h2][i] - s_delta[buf][qr]);
      }
    // dV^T[d][key] += dO^T[d][q] P[q][key];  dK^T[d][key] += Q^T[d][q] dS[q][key]
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const bf16x8 pf = frag_acc(sc[h2], 8 * g);
        const bf16x8 sf = frag_acc(dp[h2], 8 * g);
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          dv[dt] = mfma(frag_t(tdot, dt * 32, h2 * 2 + g, lane), pf, dv[dt]);
          dk[dt] = mfma(frag_t(tqt, dt * 32, h2 * 2 + g, lane), sf, dk[dt]);
        }
      }
    if (nxt < total) lstore(buf ^ 1, nxt);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }

  if (!key_ok) return;
  // Outputs: lane owns key my_key; register i of tile dt is d = 32 dt + acc_row(i).
  const int64_t off = bi * S.bstride + static_cast<int64_t>(my_key) * S.ld + hk * D;
  const int64_t doff = bi * S.d_bstride + static_cast<int64_t>(my_key) * S.d_ld + hk * D;
  constexpr int HALF_T = D / 64;   // tiles between a RoPE pair (d, d + D/2)
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) dk[dt][i] *= p.scale;
  if (S.rk) {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int d = dt * 32 + 8 * jj + 4 * (lane >> 5);
        const u32x2 rk = *reinterpret_cast<const u32x2*>(S.rk + off + d);
        const u32x2 rv = *reinterpret_cast<const u32x2*>(S.rv + off + d);
        dk[dt][4 * jj] += lo16(rk[0]);
        dk[dt][4 * jj + 1] += hi16(rk[0]);
        dk[dt][4 * jj + 2] += lo16(rk[1]);
        dk[dt][4 * jj + 3] += hi16(rk[1]);
        dv[dt][4 * jj] += lo16(rv[0]);
        dv[dt][4 * jj + 1] += hi16(rv[0]);
        dv[dt][4 * jj + 2] += lo16(rv[1]);
        dv[dt][4 * jj + 3] += hi16(rv[1]);
      }
  }
  if (S.rope) {
    const float2* tab = p.rope + static_cast<int64_t>(S.rope_row0 + my_key) * (D / 2);
#pragma unroll
    for (int dt = 0; dt < HALF_T; ++dt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int d = dt * 32 + acc_row(i, lane);
        const float2 cs = tab[d];
        const float a = dk[dt][i], b = dk[dt + HALF_T][i];
        dk[dt][i] = a * cs.x + b * cs.y;              // rotate by -angle
        dk[dt + HALF_T][i] = b * cs.x - a * cs.y;
      }
  }
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + 4 * (lane >> 5);
      *reinterpret_cast<u32x2*>(S.dk + doff + d) =
          u32x2{pack2(dk[dt][4 * jj], dk[dt][4 * jj + 1]), pack2(dk[dt][4 * jj + 2], dk[dt][4 * jj + 3])};
      *reinterpret_cast<u32x2*>(S.dv + doff + d) =
          u32x2{pack2(dv[dt][4 * jj], dv[dt][4 * jj + 1]), pack2(dv[dt][4 * jj + 2], dv[dt][4 * jj + 3])};
    }
}

// ------------------------------------------------------------------ backward: dQ
// grid: (q tiles of 128, a_t heads, b); 4 waves x 32 queries; loops over key tiles.
template <int D>
__global__ void __launch_bounds__(256) attn_bwd_dq_kernel(AttnParams p) {
  constexpr int KT = 64;
  constexpr int TILE = KT * D * 2;
  // [buf][K, K^T, V]
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][3][TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_qt = (p.n_q + 127) / 128;
  const int qt = n_qt - 1 - blockIdx.x;
  const int hq = blockIdx.y, bi = blockIdx.z;
  const int hk = hq / (p.a_t / p.k_t);
  const int q_row0 = qt * 128;
  const int my_q = q_row0 + wave * 32 + (lane & 31);
  const bool q_ok = my_q < p.n_q;
  const int my_pos = q_ok ? qpos(p.qmap, my_q) : -1;
  const int blk_last = min(q_row0 + 127, p.n_q - 1);
  const int pos_max = qpos(p.qmap, blk_last);

  bf16x8 qf[D / 16], dof[D / 16];
  {
    const int64_t off = bi * p.q_bstride + static_cast<int64_t>(my_q) * p.q_ld + hq * D;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const int dcol = (2 * kk + (lane >> 5)) * 8;
      qf[kk] = q_ok ? *reinterpret_cast<const bf16x8*>(p.q + off + dcol) : bf16x8{};
      dof[kk] = q_ok ? *reinterpret_cast<const bf16x8*>(p.dout + off + dcol) : bf16x8{};
    }
  }
  const int64_t sidx = (static_cast<int64_t>(bi) * p.a_t + hq) * p.n_q + (q_ok ? my_q : 0);
  const float my_lse = q_ok ? p.lse[sidx] * kLog2e : INFINITY;
  const float my_delta = q_ok ? p.delta[sidx] : 0.f;
  const float c = p.scale * kLog2e;
  f32x16 dq[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dq[i] = f32x16{};

  const int ntiles = total_tiles(p, KT);
  auto next_visible = [&](int from, int& seg, int& t0) {
    for (int t = from; t < ntiles; ++t) {
      if (!find_tile(p, t, KT, seg, t0)) break;
      if (p.seg[seg].pos0 + t0 <= pos_max) return t;
    }
    return ntiles;
  };
  const bool is_k = tid < 128;
  const int lt = tid & 127;
  const int tb = lt / (D / 8), dc = lt % (D / 8);
  const bool loader = tb < KT / 8;
  u32x4 stage[8];
  auto gload = [&](int seg, int t0) {
    if (!loader) return;
    const KvSeg& s = p.seg[seg];
    const uint16_t* base = (is_k ? s.k : s.v) + bi * s.bstride + hk * D;
    load8(base + static_cast<int64_t>(t0) * s.ld, s.ld, tb * 8, s.n - t0, dc * 8, stage);
  };
  auto lstore = [&](int buf) {
    if (!loader) return;
    if (is_k) {
      put_r<D>(smem[buf][0], tb * 8, dc, stage);
      put_t(smem[buf][1], tb * 8, dc, stage);
    } else {
      put_r<D>(smem[buf][2], tb * 8, dc, stage);
    }
  };

  int seg, t0;
  int cur = next_visible(0, seg, t0);
  if (cur < ntiles) {
    gload(seg, t0);
    lstore(0);
  }
  __syncthreads();
  int buf = 0;
  while (cur < ntiles) {
    const int cseg = seg, ct0 = t0;
    const int nxt = next_visible(cur + 1, seg, t0);
    if (nxt < ntiles) gload(seg, t0);
    const KvSeg& s = p.seg[cseg];
    const int kpos0 = s.pos0 + ct0;
    const int kvalid = min(KT, s.n - ct0);

    f32x16 sc[2] = {f32x16{}, f32x16{}}, dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        sc[t2] = mfma(frag_r<D>(smem[buf][0], t2 * 32, kk, lane), qf[kk], sc[t2]);
        dp[t2] = mfma(frag_r<D>(smem[buf][2], t2 * 32, kk, lane), dof[kk], dp[t2]);
      }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int kr = t2 * 32 + acc_row(i, lane);
        float pr = 0.f;
        if (q_ok && kr < kvalid && kpos0 + kr <= my_pos) pr = exp2f(sc[t2][i] * c - my_lse);
        sc[t2][i] = pr * (dp[t2][i] - my_delta);       // dS^T
      }
    // dQ^T[d][q] += K^T[d][keys] dS^T[keys][q]
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const bf16x8 sf = frag_acc(sc[t2], 8 * g);
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) dq[dt] = mfma(frag_t(smem[buf][1], dt * 32, t2 * 2 + g, lane), sf, dq[dt]);
      }
    if (nxt < ntiles) lstore(buf ^ 1);
    __syncthreads();
    buf ^= 1;
    cur = nxt;
  }
  if (!q_ok) return;
  constexpr int HALF_T = D / 64;
  const float2* tab = p.rope + static_cast<int64_t>(my_q) * (D / 2);
#pragma unroll
  for (int dt = 0; dt < HALF_T; ++dt)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int d = dt * 32 + acc_row(i, lane);
      const float2 cs = tab[d];
      const float a = dq[dt][i] * p.scale, b = dq[dt + HALF_T][i] * p.scale;
      dq[dt][i] = a * cs.x + b * cs.y;
      dq[dt + HALF_T][i] = b * cs.x - a * cs.y;
    }
  uint16_t* out = p.dq + bi * static_cast<int64_t>(p.n_q) * p.dq_ld + static_cast<int64_t>(my_q) * p.dq_ld + hq * D;
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int d = dt * 32 + 8 * jj + 4 * (lane >> 5);
      *reinterpret_cast<u32x2*>(out + d) =
          u32x2{pack2(dq[dt][4 * jj], dq[dt][4 * jj + 1]), pack2(dq[dt][4 * jj + 2], dq[dt][4 * jj + 3])};
    }
}

template <int D>
hipError_t fwd_impl(const AttnParams& p, hipStream_t stream) {
  const dim3 grid((p.n_q + 127) / 128, p.a_t, p.b);
  hipLaunchKernelGGL(attn_fwd_kernel<D>, grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

int count_blocks(const AttnParams& p, int tsz) {
  int n = 0;
  for (int s = 0; s < p.n_seg; ++s) n += (p.seg[s].n + tsz - 1) / tsz;
  return n;
}

template <int D>
hipError_t bwd_impl(const AttnParams& p, hipStream_t stream) {
  const int64_t rows = static_cast<int64_t>(p.b) * p.n_q;
  hipLaunchKernelGGL(attn_delta_kernel<D>, dim3(static_cast<unsigned>((rows + 3) / 4)), dim3(256), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<D>, dim3(count_blocks(p, 128), p.k_t, p.b), dim3(256), 0, stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_bwd_dq_kernel<D>, dim3((p.n_q + 127) / 128, p.a_t, p.b), dim3(256), 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd(const AttnParams& p, hipStream_t stream) {
  if (p.n_q <= 0) return hipSuccess;
  if (p.d_h == 128) return fwd_impl<128>(p, stream);
  if (p.d_h == 64) return fwd_impl<64>(p, stream);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd(const AttnParams& p, hipStream_t stream) {
  if (p.n_q <= 0) return hipSuccess;
  if (p.d_h == 128) return bwd_impl<128>(p, stream);
  if (p.d_h == 64) return bwd_impl<64>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace l4d
