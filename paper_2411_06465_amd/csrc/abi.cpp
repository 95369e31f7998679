// C ABI of the layer-shard library: argument validation, the exact memory
// estimate, the arena / activation-stash allocator, kernel timing, and the
// orchestration of the forward, backward and LM-head kernel sequences.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <string>
#include <vector>

#include "../../include/l4d.h"
#include "kernels.h"

using namespace l4d;

// ============================================================== errors

static thread_local std::string g_err;

static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

extern "C" const char* l4d_last_error(void) { return g_err.c_str(); }

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(L4D_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// ============================================================== kernel timing

namespace {
struct Pending {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::string g_prof_only;            // non-empty: time only the launches with this label
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_event_pool;
std::map<std::string, std::pair<int64_t, double>> g_totals;
std::vector<const char*> g_order;  // labels of the timed launches since the last reset, in launch order

hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

int drain_pending() {
  for (auto& p : g_pending) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
    if (e != hipSuccess) return fail(L4D_EDEVICE, "profile events: %s", hipGetErrorString(e));
    auto& t = g_totals[p.name];
    g_order.push_back(p.name);
    t.first += 1;
    t.second += ms;
    g_event_pool.push_back(p.a);
    g_event_pool.push_back(p.b);
  }
  g_pending.clear();
  return L4D_OK;
}

// Launch `fn` (returning hipError_t) bracketed by events when timing is on.
template <class F>
int launch(const char* name, hipStream_t s, F&& fn) {
  hipEvent_t a = nullptr, b = nullptr;
  if (g_prof_on && (g_prof_only.empty() || g_prof_only == name)) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    a = take_event();
    b = take_event();
    if (a) (void)hipEventRecord(a, s);
  }
  hipError_t e = fn();
  if (e != hipSuccess) return fail(L4D_EDEVICE, "launch of %s failed: %s", name, hipGetErrorString(e));
  if (a && b) {
    (void)hipEventRecord(b, s);
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_pending.push_back({name, a, b});
  }
  return L4D_OK;
}
}  // namespace

extern "C" int l4d_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = on != 0;
  return L4D_OK;
}

extern "C" int l4d_profile_only(const char* name) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_only = name ? name : "";
  return L4D_OK;
}

extern "C" int l4d_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  int rc = drain_pending();
  g_totals.clear();
  g_order.clear();
  return rc;
}

extern "C" int l4d_profile_read(const char* name, int64_t* launches, double* total_ms) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  int rc = drain_pending();
  if (rc) return rc;
  int64_t n = 0;
  double ms = 0;
  for (auto& kv : g_totals)
    if (!name || kv.first == name) {
      n += kv.second.first;
      ms += kv.second.second;
    }
  if (launches) *launches = n;
  if (total_ms) *total_ms = ms;
  return L4D_OK;
}

extern "C" int l4d_profile_dump(char* buf, uint64_t buf_len, uint64_t* needed) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  int rc = drain_pending();
  if (rc) return rc;
  std::string out;
  char line[256];
  for (auto& kv : g_totals) {
    snprintf(line, sizeof line, "%s %lld %.6f\n", kv.first.c_str(), (long long)kv.second.first, kv.second.second);
    out += line;
  }
  if (needed) *needed = out.size() + 1;
  if (buf && buf_len) {
    size_t n = std::min<size_t>(out.size(), buf_len - 1);
    memcpy(buf, out.data(), n);
    buf[n] = 0;
  }
  return L4D_OK;
}

extern "C" int l4d_profile_order(char* buf, uint64_t buf_len, uint64_t* needed) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  int rc = drain_pending();
  if (rc) return rc;
  std::string out;
  for (const char* n : g_order) {
    out += n;
    out += '\n';
  }
  if (needed) *needed = out.size() + 1;
  if (buf && buf_len) {
    size_t n = std::min<size_t>(out.size(), buf_len - 1);
    memcpy(buf, out.data(), n);
    buf[n] = 0;
  }
  return L4D_OK;
}

// ============================================================== memory estimate

namespace {
typedef __int128 i128;

struct Rat {  // num / den, den > 0
  i128 num, den;
};

uint64_t ceil_u64(Rat r, bool& inexact) {
  i128 q = r.num / r.den, rem = r.num % r.den;
  if (rem != 0) {
    inexact = true;
    q += 1;
  }
  return (uint64_t)q;
}

int check_model(const l4d_model* m, const l4d_parallel* p) {
  if (!m || !p) return fail(L4D_EINVAL, "model and parallel layout are required");
  if (m->hidden <= 0 || m->n_heads <= 0 || m->n_kv_heads <= 0 || m->ffn <= 0 || m->n_layers <= 0 ||
      m->vocab <= 0)
    return fail(L4D_EINVAL, "model sizes must be positive");
  if (p->seq <= 0 || p->micro_batch <= 0 || p->tp <= 0 || p->cp <= 0 || p->pp <= 0 || p->dp <= 0)
    return fail(L4D_EINVAL, "sequence, micro-batch and parallel sizes must be positive");
  if (m->hidden % m->n_heads) return fail(L4D_EINVAL, "hidden %% n_heads != 0");
  if (m->n_heads % m->n_kv_heads) return fail(L4D_EINVAL, "n_heads %% n_kv_heads != 0");
  if (m->n_heads % p->tp || m->n_kv_heads % p->tp) return fail(L4D_EINVAL, "heads not divisible by tp");
  if (m->ffn % p->tp) return fail(L4D_EINVAL, "ffn %% tp != 0");
  if (m->vocab % p->tp) return fail(L4D_EINVAL, "vocab %% tp != 0");
  if (p->seq % p->cp) return fail(L4D_EINVAL, "seq %% cp != 0");
  if (m->n_layers % p->pp) return fail(L4D_EINVAL, "n_layers %% pp != 0");
  if (p->tp_rank < 0 || p->tp_rank >= p->tp || p->cp_rank < 0 || p->cp_rank >= p->cp)
    return fail(L4D_EINVAL, "rank out of range");
  return L4D_OK;
}
}  // namespace

extern "C" int mem_estimate(const l4d_model* m, const l4d_parallel* p, l4d_mem* out) {
  int rc = check_model(m, p);
  if (rc) return rc;
  if (!out) return fail(L4D_EINVAL, "out is NULL");
  const i128 h = m->hidden, a = m->n_heads, k = m->n_kv_heads, f = m->ffn, L = m->n_layers, v = m->vocab;
  const i128 s = p->seq, b = p->micro_batch, t = p->tp, c = p->cp, pp = p->pp, d = p->dp;
  // ell * (a t) = 2h^2(a+k) + 3 h f a + 2 h a t   (Eqs. 1, 2 divided by t, plus the two norms)
  const i128 E = 2 * h * h * (a + k) + 3 * h * f * a + 2 * h * a * t;
  Rat psi;
  if (p->pp == 1) psi = {2 * h * v * a + h * a * t + L * E, a * t};   // embedding + head + final norm
  else psi = {h * v * a * pp + L * E, a * t * pp};                   // first stage (Eq. 7)
  bool inexact = false;
  out->params_per_gpu = ceil_u64(psi, inexact);
  out->weight_bytes = ceil_u64({2 * psi.num, psi.den}, inexact);
  out->grad_bytes = ceil_u64({4 * psi.num, psi.den}, inexact);
  out->optim_bytes = ceil_u64({12 * psi.num, psi.den * d * c}, inexact);
  // per layer: s b (12 a h + 4 k h + 8 f a) / (t c a)     (Eq. 12 / (tc))
  const i128 lay = 12 * a * h + 4 * k * h + 8 * f * a;
  out->act_bytes_per_layer = ceil_u64({s * b * lay, t * c * a}, inexact);
  // Eq. 17: s b [L lay + 8 p a h + [p=1] 4 a (h + v)] / (t c a)
  i128 act = L * lay + 8 * pp * a * h;
  if (p->pp == 1) act += 4 * a * (h + v);
  out->act_bytes = ceil_u64({s * b * act, t * c * a}, inexact);
  out->total_bytes = out->weight_bytes + out->grad_bytes + out->optim_bytes + out->act_bytes;
  out->inexact = inexact ? 1u : 0u;
  return L4D_OK;
}

extern "C" int mem_fit(const l4d_mem* est, uint64_t device_bytes, int* fit) {
  if (!est || !fit || device_bytes == 0) return fail(L4D_EINVAL, "est, fit and device_bytes are required");
  // total <= 0.8 M  <=>  5 total <= 4 M, in 128-bit integers
  const unsigned __int128 t5 = (unsigned __int128)est->total_bytes * 5, m4 = (unsigned __int128)device_bytes * 4;
  *fit = t5 <= m4 ? L4D_FITS : (est->total_bytes <= device_bytes ? L4D_NEAR_LIMIT : L4D_OOM);
  return L4D_OK;
}

// ============================================================== arena

struct l4d_arena {
  uintptr_t base;
  uint64_t cap;
  std::map<uint64_t, uint64_t> free_;  // offset -> size
  uint64_t in_use = 0, peak = 0;
  std::set<const l4d_stash*> live;
};

namespace {
constexpr uint64_t kAlign = 256;
uint64_t align_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool arena_alloc(l4d_arena* A, uint64_t size, uint64_t* off) {
  size = align_up(std::max<uint64_t>(size, 1));
  for (auto it = A->free_.begin(); it != A->free_.end(); ++it) {
    if (it->second >= size) {
      *off = it->first;
      uint64_t rest = it->second - size, roff = it->first + size;
      A->free_.erase(it);
      if (rest) A->free_[roff] = rest;
      A->in_use += size;
      A->peak = std::max(A->peak, A->in_use);
      return true;
    }
  }
  return false;
}

void arena_free(l4d_arena* A, uint64_t off, uint64_t size) {
  size = align_up(std::max<uint64_t>(size, 1));
  A->in_use -= size;
  auto it = A->free_.emplace(off, size).first;
  auto nx = std::next(it);
  if (nx != A->free_.end() && it->first + it->second == nx->first) {
    it->second += nx->second;
    A->free_.erase(nx);
  }
  if (it != A->free_.begin()) {
    auto pv = std::prev(it);
    if (pv->first + pv->second == it->first) {
      pv->second += it->second;
      A->free_.erase(it);
    }
  }
}

// A transient workspace: a list of sub-buffers carved from one arena block.
struct Workspace {
  l4d_arena* A = nullptr;
  uint64_t off = 0, size = 0;
  bool held = false;
  ~Workspace() {
    if (held) arena_free(A, off, size);
  }
};

struct Carver {  // bump-allocates aligned pieces of a byte range
  uint64_t used = 0;
  uint64_t take(uint64_t bytes) {
    uint64_t o = used;
    used += align_up(bytes);
    return o;
  }
};
}  // namespace

extern "C" int l4d_arena_create(void* dev_base, uint64_t capacity, l4d_arena** out) {
  if (!out) return fail(L4D_EINVAL, "out is NULL");
  if (!dev_base && capacity) return fail(L4D_EINVAL, "dev_base is NULL");
  if (reinterpret_cast<uintptr_t>(dev_base) % kAlign) return fail(L4D_EINVAL, "dev_base must be 256-byte aligned");
  auto* A = new l4d_arena();
  A->base = reinterpret_cast<uintptr_t>(dev_base);
  A->cap = capacity / kAlign * kAlign;
  if (A->cap) A->free_[0] = A->cap;
  *out = A;
  return L4D_OK;
}

extern "C" int l4d_arena_destroy(l4d_arena* A) {
  if (!A) return L4D_OK;
  if (!A->live.empty()) return fail(L4D_EINVAL, "arena still holds %zu live stash(es)", A->live.size());
  delete A;
  return L4D_OK;
}

extern "C" int l4d_arena_stats(const l4d_arena* A, uint64_t* in_use, uint64_t* peak, uint64_t* capacity) {
  if (!A) return fail(L4D_EINVAL, "arena is NULL");
  if (in_use) *in_use = A->in_use;
  if (peak) *peak = A->peak;
  if (capacity) *capacity = A->cap;
  return L4D_OK;
}

// ============================================================== shard geometry

namespace {
struct Shard {
  int64_t h, a, k, f, s, b, t, c, tr, cr;
  int64_t d, a_t, k_t, f_t, s_c, s_sp;
  float eps, base;
  ChunkMap qmap;
  int n_remote_runs;
  int64_t rem_chunk_start[4], rem_chunk_count[4];  // runs of consecutive remote chunks (chunk ids)
  int64_t chunk_len;
};

int make_shard(const l4d_model* m, const l4d_parallel* p, Shard* S) {
  int rc = check_model(m, p);
  if (rc) return rc;
  Shard& x = *S;
  x.h = m->hidden; x.a = m->n_heads; x.k = m->n_kv_heads; x.f = m->ffn;
  x.s = p->seq; x.b = p->micro_batch; x.t = p->tp; x.c = p->cp; x.tr = p->tp_rank; x.cr = p->cp_rank;
  x.eps = m->rms_eps; x.base = m->rope_base;
  x.d = x.h / x.a; x.a_t = x.a / x.t; x.k_t = x.k / x.t; x.f_t = x.f / x.t;
  x.s_c = x.s / x.c;
  if (x.s_c % x.t) return fail(L4D_EINVAL, "local sequence %lld not divisible by tp", (long long)x.s_c);
  x.s_sp = x.s_c / x.t;
  if (x.d != 64 && x.d != 128) return fail(L4D_EINVAL, "head dim %lld unsupported (64 or 128)", (long long)x.d);
  if (x.h % 8 || x.f_t % 8) return fail(L4D_EINVAL, "hidden and ffn/tp must be multiples of 8");
  if (x.h > 8192) return fail(L4D_EINVAL, "hidden > 8192 unsupported");
  if (x.c > 1 && x.s % (2 * x.c)) return fail(L4D_EINVAL, "seq %% (2 cp) != 0");
  if (x.b * x.s_c > (int64_t)1 << 30 || x.h * x.s > (int64_t)1 << 40)
    return fail(L4D_EINVAL, "problem too large");
  // CP layout: 2c chunks, rank r owns r and 2c-1-r (Sec. 2.1 / 3.2.3 load-balanced reading)
  if (x.c == 1) {
    x.chunk_len = x.s;
    x.qmap = ChunkMap{1, (int32_t)x.s, {0, 0}};
    x.n_remote_runs = 0;
  } else {
    x.chunk_len = x.s / (2 * x.c);
    x.qmap = ChunkMap{2, (int32_t)x.chunk_len, {(int32_t)x.cr, (int32_t)(2 * x.c - 1 - x.cr)}};
    x.n_remote_runs = 0;
    int64_t i = 0;
    while (i < 2 * x.c) {
      if (i == x.cr || i == 2 * x.c - 1 - x.cr) { ++i; continue; }
      int64_t j = i;
      while (j + 1 < 2 * x.c && j + 1 != x.cr && j + 1 != 2 * x.c - 1 - x.cr) ++j;
      x.rem_chunk_start[x.n_remote_runs] = i;
      x.rem_chunk_count[x.n_remote_runs] = j - i + 1;
      ++x.n_remote_runs;
      i = j + 1;
    }
  }
  return L4D_OK;
}

int64_t qkv_cols(const Shard& x) { return (x.a_t + 2 * x.k_t) * x.d; }
}  // namespace

// ============================================================== stash

enum StashKind { kLayerStash = 0, kHeadStash = 1, kEmbStash = 2 };

struct l4d_stash {
  l4d_arena* arena;
  uint64_t block_off, block_size;
  uint64_t off[L4D_STASH_COUNT], bytes[L4D_STASH_COUNT];
  uint64_t formula, aux, padding;
  Shard shape;
  int kind = kLayerStash;
  int count = L4D_STASH_COUNT;
};

namespace {
void stash_sizes(const Shard& x, uint64_t* bytes) {
  const uint64_t sp = x.b * x.s_sp * x.h * 2, tok = x.b * x.s_c;
  bytes[L4D_STASH_X] = bytes[L4D_STASH_XN1] = bytes[L4D_STASH_H1] = bytes[L4D_STASH_XN2] = sp;
  bytes[L4D_STASH_Q] = bytes[L4D_STASH_CTX] = tok * x.a_t * x.d * 2;
  bytes[L4D_STASH_K] = bytes[L4D_STASH_V] = tok * x.k_t * x.d * 2;
  bytes[L4D_STASH_GATE] = bytes[L4D_STASH_UP] = bytes[L4D_STASH_ACT] = bytes[L4D_STASH_PROD] = tok * x.f_t * 2;
  bytes[L4D_STASH_LSE] = x.b * x.a_t * x.s_c * 4;
}

// One arena block holding `count` tensors of the given sizes, 256-byte aligned;
// the tensor `aux_slot` (or none, -1) is reported as aux, the rest as formula.
int stash_reserve_sized(l4d_arena* A, const Shard& x, int kind, int count, const uint64_t* bytes, int aux_slot,
                        l4d_stash** out) {
  auto* st = new l4d_stash();
  st->arena = A;
  st->shape = x;
  st->kind = kind;
  st->count = count;
  uint64_t total = 0, raw = 0;
  for (int i = 0; i < count; ++i) {
    st->bytes[i] = bytes[i];
    st->off[i] = total;
    total += align_up(st->bytes[i]);
    if (i != aux_slot) raw += st->bytes[i];
  }
  st->formula = raw;
  st->aux = aux_slot >= 0 ? st->bytes[aux_slot] : 0;
  st->padding = total - raw - st->aux;
  if (!arena_alloc(A, total, &st->block_off)) {
    delete st;
    return fail(L4D_ENOMEM, "stash needs %llu bytes; arena has %llu of %llu in use", (unsigned long long)total,
                (unsigned long long)A->in_use, (unsigned long long)A->cap);
  }
  st->block_size = total;
  A->live.insert(st);
  *out = st;
  return L4D_OK;
}

int stash_reserve(l4d_arena* A, const Shard& x, l4d_stash** out) {
  uint64_t bytes[L4D_STASH_COUNT];
  stash_sizes(x, bytes);
  return stash_reserve_sized(A, x, kLayerStash, L4D_STASH_COUNT, bytes, L4D_STASH_LSE, out);
}

template <class T = uint16_t>
T* sptr(const l4d_stash* st, int which) {
  return reinterpret_cast<T*>(st->arena->base + st->block_off + st->off[which]);
}
}  // namespace

extern "C" int l4d_stash_reserve(l4d_arena* A, const l4d_model* m, const l4d_parallel* p, l4d_stash** out) {
  if (!A || !out) return fail(L4D_EINVAL, "arena and out are required");
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  return stash_reserve(A, x, out);
}

extern "C" int l4d_stash_bytes(const l4d_stash* st, uint64_t* formula, uint64_t* aux, uint64_t* padding) {
  if (!st) return fail(L4D_EINVAL, "stash is NULL");
  if (formula) *formula = st->formula;
  if (aux) *aux = st->aux;
  if (padding) *padding = st->padding;
  return L4D_OK;
}

extern "C" int l4d_stash_tensor(const l4d_stash* st, int which, void** ptr, uint64_t* bytes) {
  if (!st) return fail(L4D_EINVAL, "stash is NULL");
  if (which < 0 || which >= st->count) return fail(L4D_EINVAL, "no stash tensor %d", which);
  if (ptr) *ptr = sptr<void>(st, which);
  if (bytes) *bytes = st->bytes[which];
  return L4D_OK;
}

extern "C" int l4d_stash_release(l4d_arena* A, l4d_stash* st) {
  if (!A || !st) return fail(L4D_EINVAL, "arena and stash are required");
  if (st->arena != A || !A->live.count(st)) return fail(L4D_EINVAL, "stash does not belong to this arena");
  arena_free(A, st->block_off, st->block_size);
  A->live.erase(st);
  delete st;
  return L4D_OK;
}

// ============================================================== workspace plans

namespace {
struct FwdWs {
  uint64_t rope, o_send, ffn_send, total;
};
struct BwdWs {
  uint64_t rope, dgu, dxn2, dh1, dh1_f32, dctx, delta, dqkv, dxn1, partial, dxn2_send, dxn1_send, dkv, dwpart, total;
};

uint64_t split_ws_bytes(int64_t M, int64_t N, int64_t K, bool acc_f32 = true) {
  const int s = gemm_ksplits(M, N, K, acc_f32);
  return s <= 1 ? 0 : (uint64_t)(acc_f32 ? s - 1 : s) * M * N * 4;
}

FwdWs plan_fwd(const Shard& x, const l4d_peer_outputs* sends) {
  Carver cv;
  FwdWs w;
  const uint64_t peer_rows = x.b * (x.t - 1) * x.s_sp * x.h * 2;
  w.rope = cv.take(x.s_c * (x.d / 2) * 8);
  w.o_send = (x.t > 1 && !(sends && sends->o_partial)) ? cv.take(peer_rows) : 0;
  w.ffn_send = (x.t > 1 && !(sends && sends->ffn_partial)) ? cv.take(peer_rows) : 0;
  w.total = cv.used;
  return w;
}

BwdWs plan_bwd(const Shard& x, const l4d_peer_outputs* sends) {
  Carver cv;
  BwdWs w;
  const uint64_t tok = x.b * x.s_c, sp = x.b * x.s_sp * x.h * 2;
  const uint64_t peer_rows = x.b * (x.t - 1) * x.s_sp * x.h * 2;
  w.rope = cv.take(x.s_c * (x.d / 2) * 8);
  w.dgu = cv.take(tok * 2 * x.f_t * 2);
  w.dxn2 = cv.take(2 * sp);       // fp32: only the norm backward reads it
  w.dh1 = cv.take(sp);            // bf16: operand of the output-projection products
  w.dh1_f32 = cv.take(2 * sp);    // fp32: the residual the norm-1 backward adds
  w.dctx = cv.take(tok * x.a_t * x.d * 2);
  w.delta = cv.take(x.b * x.a_t * x.s_c * 4);
  w.dqkv = cv.take(tok * qkv_cols(x) * 2);
  w.dxn1 = cv.take(2 * sp);       // fp32
  w.partial = cv.take((uint64_t)rmsnorm_bwd_partials(x.b * x.s_sp) * x.h * 4);
  w.dxn2_send = (x.t > 1 && !(sends && sends->dxn2_partial)) ? cv.take(peer_rows) : 0;
  w.dxn1_send = (x.t > 1 && !(sends && sends->dxn1_partial)) ? cv.take(peer_rows) : 0;
  // fp32 dK/dV partials when the query heads of a kv-head are split (at most a/k slices)
  const int64_t group = x.a / x.k;
  w.dkv = group > 1 ? cv.take(2 * (uint64_t)group * x.b * x.s * x.k_t * x.d * 4) : 0;
  // fp32 partials of the weight-gradient GEMMs that split their K (token) range
  const int64_t tk = (int64_t)tok;
  const uint64_t dwp = std::max({split_ws_bytes(x.h, x.f_t, tk), split_ws_bytes(2 * x.f_t, x.h, tk),
                                 split_ws_bytes(x.h, x.a_t * x.d, tk), split_ws_bytes(qkv_cols(x), x.h, tk),
                                 split_ws_bytes(tk, x.a_t * x.d, x.h, false)});   // and the O dX GEMM
  w.dwpart = dwp ? cv.take(dwp) : 0;
  w.total = cv.used;
  return w;
}

int take_ws(l4d_arena* A, uint64_t bytes, Workspace& ws) {
  ws.A = A;
  ws.size = bytes;
  if (!arena_alloc(A, bytes, &ws.off))
    return fail(L4D_ENOMEM, "workspace needs %llu bytes; arena has %llu of %llu in use", (unsigned long long)bytes,
                (unsigned long long)A->in_use, (unsigned long long)A->cap);
  ws.held = true;
  return L4D_OK;
}
}  // namespace

extern "C" int l4d_layer_workspace_bytes(const l4d_model* m, const l4d_parallel* p, uint64_t* fwd, uint64_t* bwd) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  if (fwd) *fwd = align_up(plan_fwd(x, nullptr).total);
  if (bwd) *bwd = align_up(plan_bwd(x, nullptr).total);
  return L4D_OK;
}

namespace {
// A K-contiguous x N-contiguous GEMM whose K is long but not a multiple of 128
// (the LM head's d_hidden over a vocabulary shard) runs its first K - K % 128 on
// the BK = 64 kernel and the rest on the ragged-K kernel, summing in fp32.
bool ragged_k_split(int64_t K) { return K % 128 != 0 && K >= 1024; }
}  // namespace

extern "C" int l4d_lm_head_workspace_bytes(int64_t n, int64_t h, int64_t v_t, uint64_t* bytes) {
  if (n < 0 || h <= 0 || v_t <= 0) return fail(L4D_EINVAL, "bad LM-head sizes");
  if (bytes) *bytes = align_up((uint64_t)n * v_t * 2) + (ragged_k_split(v_t) ? align_up((uint64_t)n * h * 4) : 0);
  return L4D_OK;
}

// ============================================================== layer helpers

namespace {
inline RowSrc gathered(const void* own, const void* peer, const Shard& x) {
  if (x.t == 1) return RowSrc::plain(own, x.h);
  return RowSrc{static_cast<const uint16_t*>(own), static_cast<const uint16_t*>(peer), x.h, (int32_t)x.s_c,
                (int32_t)x.s_sp, (int32_t)x.tr, (int32_t)x.t};
}

inline Operand op(RowSrc src, int64_t rows) { return Operand{src, (int32_t)rows, 0, 0}; }

inline EpiParams epi_residual(const Shard& x, uint16_t* own_out, const void* resid, const void* receipt,
                              void* send, float* own_out_f32 = nullptr) {
  EpiParams e{};
  e.kind = EpiKind::ResidualSP;
  e.ldc = x.h;
  e.own_out = own_out;
  e.own_out_f32 = own_out_f32;
  e.resid = static_cast<const uint16_t*>(resid);
  e.receipt = static_cast<const uint16_t*>(receipt);
  e.send = static_cast<uint16_t*>(send);
  e.s_c = (int32_t)x.s_c;
  e.s_sp = (int32_t)x.s_sp;
  e.r = (int32_t)x.tr;
  e.t = (int32_t)x.t;
  return e;
}

inline EpiParams epi_acc(float* c, int64_t ldc) {
  EpiParams e{};
  e.kind = EpiKind::AccF32;
  e.c = c;
  e.ldc = ldc;
  return e;
}

inline EpiParams epi_store(void* c, int64_t ldc) {
  EpiParams e{};
  e.kind = EpiKind::StoreBF16;
  e.c = c;
  e.ldc = ldc;
  return e;
}

// split_ws: room for the fp32 partials of a split K range (AccF32 only; NULL =
// never split); split_ws_bytes(M, N, K) bytes are needed.
int run_gemm(const char* name, hipStream_t s, int64_t M, int64_t N, int64_t K, Operand A, Layout la, Operand B,
             Layout lb, EpiParams e, float* split_ws = nullptr) {
  GemmParams p{};
  p.M = (int32_t)M;
  p.N = (int32_t)N;
  p.K = (int32_t)K;
  p.A = A;
  p.B = B;
  p.epi = e;
  const bool acc = e.kind == EpiKind::AccF32;
  if ((acc || e.kind == EpiKind::StoreBF16) && split_ws) {
    p.k_splits = gemm_ksplits(M, N, K, acc);
    p.partial = split_ws;
  }
  int rc = launch(name, s, [&] { return gemm(p, la, lb, s); });
  if (rc || p.k_splits <= 1) return rc;
  return launch("gemm_splitk_reduce", s, [&] {
    return acc ? gemm_split_reduce(static_cast<float*>(e.c), e.ldc, split_ws, M, N, p.k_splits, s)
               : gemm_split_store(static_cast<uint16_t*>(e.c), e.ldc, split_ws, M, N, p.k_splits, s);
  });
}

// Key runs of the attention: local chunks (stash K/V) then remote runs.
void key_segments(const Shard& x, AttnParams& ap, const uint16_t* K, const uint16_t* V, const uint16_t* rK,
                  const uint16_t* rV, uint16_t* dqkv, uint16_t* d_rk, uint16_t* d_rv, const uint16_t* cp_dk,
                  const uint16_t* cp_dv) {
  const int64_t kvw = x.k_t * x.d, qc = qkv_cols(x);
  ap.n_seg = 0;
  const int n_local = x.c == 1 ? 1 : 2;
  const int64_t run = x.c == 1 ? x.s : x.chunk_len;
  for (int i = 0; i < n_local; ++i) {
    KvSeg& g = ap.seg[ap.n_seg++];
    g = KvSeg{};
    const int64_t row0 = i * run;
    g.k = K + row0 * kvw;
    g.v = V + row0 * kvw;
    g.ld = kvw;
    g.bstride = x.s_c * kvw;
    if (dqkv) {
      g.dk = dqkv + row0 * qc + x.a_t * x.d;
      g.dv = dqkv + row0 * qc + (x.a_t + x.k_t) * x.d;
      g.d_ld = qc;
      g.d_bstride = x.s_c * qc;
    }
    if (cp_dk) {
      g.rk = cp_dk + row0 * kvw;
      g.rv = cp_dv + row0 * kvw;
    }
    g.n = (int32_t)run;
    g.pos0 = (int32_t)(x.qmap.chunk_id[i] * x.qmap.chunk_len);
    g.rope = 1;
    g.rope_row0 = (int32_t)row0;
  }
  int64_t rrow = 0;
  const int64_t rem_tokens = x.s - x.s_c;
  for (int r = 0; r < x.n_remote_runs; ++r) {
    KvSeg& g = ap.seg[ap.n_seg++];
    g = KvSeg{};
    const int64_t n = x.rem_chunk_count[r] * x.chunk_len;
    g.k = rK + rrow * kvw;
    g.v = rV + rrow * kvw;
    g.ld = kvw;
    g.bstride = rem_tokens * kvw;
    if (d_rk) {
      g.dk = d_rk + rrow * kvw;
      g.dv = d_rv + rrow * kvw;
      g.d_ld = kvw;
      g.d_bstride = rem_tokens * kvw;
    }
    g.n = (int32_t)n;
    g.pos0 = (int32_t)(x.rem_chunk_start[r] * x.chunk_len);
    g.rope = 0;
    rrow += n;
  }
}

AttnParams attn_params(const Shard& x) {
  AttnParams ap{};
  ap.n_split = 1;
  ap.b = (int32_t)x.b;
  ap.a_t = (int32_t)x.a_t;
  ap.k_t = (int32_t)x.k_t;
  ap.d_h = (int32_t)x.d;
  ap.n_q = (int32_t)x.s_c;
  ap.q_ld = x.a_t * x.d;
  ap.q_bstride = x.s_c * x.a_t * x.d;
  ap.qmap = x.qmap;
  ap.scale = 1.0f / std::sqrt((float)x.d);
  return ap;
}

int check_peers(const Shard& x, const l4d_peer_inputs* pi, bool bwd) {
  if (x.c > 1 && (!pi || !pi->remote_k || !pi->remote_v))
    return fail(L4D_EINVAL, "cp > 1 needs remote_k and remote_v");
  if (x.t > 1) {
    if (!pi || !pi->sp_peer_xn1 || !pi->sp_peer_xn2)
      return fail(L4D_EINVAL, "tp > 1 needs sp_peer_xn1 and sp_peer_xn2");
    if (bwd && (!pi->sp_peer_dy || !pi->sp_peer_dh1))
      return fail(L4D_EINVAL, "tp > 1 backward needs sp_peer_dy and sp_peer_dh1");
  }
  if (x.c > 1 && pi && ((pi->cp_peer_dk == nullptr) != (pi->cp_peer_dv == nullptr)))
    return fail(L4D_EINVAL, "cp_peer_dk and cp_peer_dv go together");
  return L4D_OK;
}
}  // namespace

// ============================================================== layer forward

extern "C" int llama_layer_fwd(const l4d_model* m, const l4d_parallel* p, const l4d_layer_weights* w,
                               const void* x_in, const l4d_peer_inputs* peers, const l4d_peer_outputs* sends,
                               void* y, l4d_arena* A, l4d_stash** stash_out, void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  if (!w || !w->norm1 || !w->qkv || !w->o || !w->norm2 || !w->gate_up || !w->down)
    return fail(L4D_EINVAL, "all six weights are required");
  if (!x_in || !y || !A || !stash_out) return fail(L4D_EINVAL, "x, y, arena and stash_out are required");
  if ((rc = check_peers(x, peers, false))) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);

  const FwdWs plan = plan_fwd(x, sends);
  l4d_stash* st = nullptr;
  if ((rc = stash_reserve(A, x, &st))) return rc;
  Workspace ws;
  if ((rc = take_ws(A, plan.total, ws))) {
    l4d_stash_release(A, st);
    return rc;
  }
  uint8_t* wsb = reinterpret_cast<uint8_t*>(A->base + ws.off);
  float2* rope = reinterpret_cast<float2*>(wsb + plan.rope);
  const l4d_peer_inputs none{};
  const l4d_peer_inputs& pi = peers ? *peers : none;
  void* o_send = (sends && sends->o_partial) ? sends->o_partial : (void*)(wsb + plan.o_send);
  void* ffn_send = (sends && sends->ffn_partial) ? sends->ffn_partial : (void*)(wsb + plan.ffn_send);
  const int64_t tok = x.b * x.s_c, nq = x.a_t * x.d, nk = x.k_t * x.d;

  auto body = [&]() -> int {
    int r;
    if ((r = launch("rope_table", s, [&] { return rope_table(rope, x.qmap, (int32_t)x.s_c, (int32_t)x.d, x.base, s); })))
      return r;
    // norm-1, stashing its input x as it goes
    if ((r = launch("rmsnorm1_fwd", s, [&] {
           return rmsnorm_fwd(static_cast<const uint16_t*>(x_in), static_cast<const uint16_t*>(w->norm1),
                              sptr(st, L4D_STASH_XN1), x.b * x.s_sp, (int32_t)x.h, x.eps, s, sptr(st, L4D_STASH_X));
         })))
      return r;
    // [Q|K|V] = xn1_full W_qkv^T, RoPE on Q, K
    EpiParams eq{};
    eq.kind = EpiKind::QkvRope;
    eq.q = sptr(st, L4D_STASH_Q);
    eq.k = sptr(st, L4D_STASH_K);
    eq.v = sptr(st, L4D_STASH_V);
    eq.nq = (int32_t)nq;
    eq.nk = (int32_t)nk;
    eq.rope = rope;
    eq.d_h = (int32_t)x.d;
    eq.s_c = (int32_t)x.s_c;
    if ((r = run_gemm("gemm_qkv", s, tok, qkv_cols(x), x.h, op(gathered(sptr(st, L4D_STASH_XN1), pi.sp_peer_xn1, x), tok),
                      Layout::KC, op(RowSrc::plain(w->qkv, x.h), qkv_cols(x)), Layout::KC, eq)))
      return r;
    // attention
    AttnParams ap = attn_params(x);
    ap.q = sptr(st, L4D_STASH_Q);
    ap.o = sptr(st, L4D_STASH_CTX);
    ap.lse = sptr<float>(st, L4D_STASH_LSE);
    key_segments(x, ap, sptr(st, L4D_STASH_K), sptr(st, L4D_STASH_V), static_cast<const uint16_t*>(pi.remote_k),
                 static_cast<const uint16_t*>(pi.remote_v), nullptr, nullptr, nullptr, nullptr, nullptr);
    if ((r = launch("attn_fwd", s, [&] { return attn_fwd(ap, s); }))) return r;
    // h1 = x + ctx W_o^T (own rows; peers' rows are sent)
    if ((r = run_gemm("gemm_o", s, tok, x.h, nq, op(RowSrc::plain(sptr(st, L4D_STASH_CTX), nq), tok), Layout::KC,
                      op(RowSrc::plain(w->o, nq), x.h), Layout::KC,
                      epi_residual(x, sptr(st, L4D_STASH_H1), x_in, pi.sp_peer_o, o_send))))
      return r;
    if ((r = launch("rmsnorm2_fwd", s, [&] {
           return rmsnorm_fwd(sptr(st, L4D_STASH_H1), static_cast<const uint16_t*>(w->norm2), sptr(st, L4D_STASH_XN2),
                              x.b * x.s_sp, (int32_t)x.h, x.eps, s);
         })))
      return r;
    // [G|U] = xn2_full W_gu^T with the SwiGLU epilogue
    EpiParams eg{};
    eg.kind = EpiKind::SwiGLUFwd;
    eg.g_out = sptr(st, L4D_STASH_GATE);
    eg.u_out = sptr(st, L4D_STASH_UP);
    eg.act_out = sptr(st, L4D_STASH_ACT);
    eg.prod_out = sptr(st, L4D_STASH_PROD);
    eg.f = (int32_t)x.f_t;
    Operand bgu{RowSrc::plain(w->gate_up, x.h), (int32_t)(2 * x.f_t), (int32_t)x.f_t, x.f_t};
    if ((r = run_gemm("gemm_gate_up", s, tok, 2 * x.f_t, x.h, op(gathered(sptr(st, L4D_STASH_XN2), pi.sp_peer_xn2, x), tok),
                      Layout::KC, bgu, Layout::KC, eg)))
      return r;
    // y = h1 + prod W_down^T
    if ((r = run_gemm("gemm_down", s, tok, x.h, x.f_t, op(RowSrc::plain(sptr(st, L4D_STASH_PROD), x.f_t), tok),
                      Layout::KC, op(RowSrc::plain(w->down, x.f_t), x.h), Layout::KC,
                      epi_residual(x, static_cast<uint16_t*>(y), sptr(st, L4D_STASH_H1), pi.sp_peer_ffn, ffn_send))))
      return r;
    return L4D_OK;
  };
  rc = body();
  if (rc) {
    l4d_stash_release(A, st);
    return rc;
  }
  *stash_out = st;
  return L4D_OK;
}

// ============================================================== layer backward

extern "C" int llama_layer_bwd(const l4d_model* m, const l4d_parallel* p, const l4d_layer_weights* w,
                               const l4d_peer_inputs* peers, const l4d_peer_outputs* sends, l4d_stash* st,
                               const void* dy, void* dx, const l4d_layer_grads* dw, void* d_remote_k,
                               void* d_remote_v, l4d_arena* A, void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  if (!w || !w->norm1 || !w->qkv || !w->o || !w->norm2 || !w->gate_up || !w->down)
    return fail(L4D_EINVAL, "all six weights are required");
  if (!dw || !dw->norm1 || !dw->qkv || !dw->o || !dw->norm2 || !dw->gate_up || !dw->down)
    return fail(L4D_EINVAL, "all six gradient accumulators are required");
  if (!st || !A || !dy || !dx) return fail(L4D_EINVAL, "stash, arena, dy and dx are required");
  if (st->arena != A || !A->live.count(st)) return fail(L4D_EINVAL, "stash does not belong to this arena");
  if (st->kind != kLayerStash) return fail(L4D_EINVAL, "not a layer stash");
  const Shard& sx = st->shape;
  if (sx.h != x.h || sx.a != x.a || sx.k != x.k || sx.f != x.f || sx.s != x.s || sx.b != x.b || sx.t != x.t ||
      sx.c != x.c || sx.tr != x.tr || sx.cr != x.cr)
    return fail(L4D_EINVAL, "stash was made for another shape");
  if (x.c > 1 && (!d_remote_k || !d_remote_v)) return fail(L4D_EINVAL, "cp > 1 needs d_remote_k and d_remote_v");
  if ((rc = check_peers(x, peers, true))) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);

  const BwdWs plan = plan_bwd(x, sends);
  Workspace ws;
  if ((rc = take_ws(A, plan.total, ws))) return rc;
  uint8_t* wsb = reinterpret_cast<uint8_t*>(A->base + ws.off);
  auto W = [&](uint64_t off) { return reinterpret_cast<uint16_t*>(wsb + off); };
  float2* rope = reinterpret_cast<float2*>(wsb + plan.rope);
  uint16_t *dgu = W(plan.dgu), *dh1 = W(plan.dh1), *dctx = W(plan.dctx), *dqkv = W(plan.dqkv);
  auto F = [&](uint64_t off) { return reinterpret_cast<float*>(wsb + off); };
  float *dxn2 = F(plan.dxn2), *dxn1 = F(plan.dxn1), *dh1_f32 = F(plan.dh1_f32);
  float* delta = reinterpret_cast<float*>(wsb + plan.delta);
  float* partial = reinterpret_cast<float*>(wsb + plan.partial);
  float* dwpart = plan.dwpart ? reinterpret_cast<float*>(wsb + plan.dwpart) : nullptr;
  const l4d_peer_inputs none{};
  const l4d_peer_inputs& pi = peers ? *peers : none;
  void* dxn2_send = (sends && sends->dxn2_partial) ? sends->dxn2_partial : (void*)W(plan.dxn2_send);
  void* dxn1_send = (sends && sends->dxn1_partial) ? sends->dxn1_partial : (void*)W(plan.dxn1_send);
  const int64_t tok = x.b * x.s_c, nq = x.a_t * x.d, qc = qkv_cols(x), rows_sp = x.b * x.s_sp;
  const int32_t npart = rmsnorm_bwd_partials(rows_sp);

  auto body = [&]() -> int {
    int r;
    if ((r = launch("rope_table", s, [&] { return rope_table(rope, x.qmap, (int32_t)x.s_c, (int32_t)x.d, x.base, s); })))
      return r;
    const RowSrc dy_full = gathered(dy, pi.sp_peer_dy, x);
    // d(prod) = dy_full W_down, consumed by the SwiGLU backward in the epilogue
    EpiParams es{};
    es.kind = EpiKind::SwiGLUBwd;
    es.g_in = sptr(st, L4D_STASH_GATE);
    es.u_in = sptr(st, L4D_STASH_UP);
    es.act_in = sptr(st, L4D_STASH_ACT);
    es.dgu = dgu;
    es.f = (int32_t)x.f_t;
    if ((r = run_gemm("gemm_down_dx", s, tok, x.f_t, x.h, op(dy_full, tok), Layout::KC,
                      op(RowSrc::plain(w->down, x.f_t), x.f_t), Layout::MN, es)))
      return r;
    // dW_down += dy_full^T prod
    if ((r = run_gemm("gemm_down_dw", s, x.h, x.f_t, tok, op(dy_full, x.h), Layout::MN,
                      op(RowSrc::plain(sptr(st, L4D_STASH_PROD), x.f_t), x.f_t), Layout::MN, epi_acc(dw->down, x.f_t), dwpart)))
      return r;
    // d(xn2) = dGU W_gu (own rows + receipt; peers' rows sent)
    if ((r = run_gemm("gemm_gate_up_dx", s, tok, x.h, 2 * x.f_t, op(RowSrc::plain(dgu, 2 * x.f_t), tok), Layout::KC,
                      op(RowSrc::plain(w->gate_up, x.h), x.h), Layout::MN,
                      epi_residual(x, nullptr, nullptr, pi.sp_peer_dxn2, dxn2_send, dxn2))))
      return r;
    const RowSrc xn2_full = gathered(sptr(st, L4D_STASH_XN2), pi.sp_peer_xn2, x);
    if ((r = run_gemm("gemm_gate_up_dw", s, 2 * x.f_t, x.h, tok, op(RowSrc::plain(dgu, 2 * x.f_t), 2 * x.f_t),
                      Layout::MN, op(xn2_full, x.h), Layout::MN, epi_acc(dw->gate_up, x.h), dwpart)))
      return r;
    // norm-2 backward + residual: dh1 in bf16 (product operand) and fp32 (residual of dx)
    if ((r = launch("rmsnorm2_bwd", s, [&] {
           const NormBwdIo io{nullptr, dxn2, static_cast<const uint16_t*>(dy), nullptr, dh1, dh1_f32};
           return rmsnorm_bwd(sptr(st, L4D_STASH_H1), static_cast<const uint16_t*>(w->norm2), io, partial, npart,
                              rows_sp, (int32_t)x.h, x.eps, s);
         })))
      return r;
    if ((r = launch("reduce_gain", s, [&] { return reduce_rows_add(partial, npart, (int32_t)x.h, dw->norm2, s); })))
      return r;
    // attention output projection
    const RowSrc dh1_full = gathered(dh1, pi.sp_peer_dh1, x);
    if ((r = run_gemm("gemm_o_dx", s, tok, nq, x.h, op(dh1_full, tok), Layout::KC, op(RowSrc::plain(w->o, nq), nq),
                      Layout::MN, epi_store(dctx, nq), dwpart)))
      return r;
    if ((r = run_gemm("gemm_o_dw", s, x.h, nq, tok, op(dh1_full, x.h), Layout::MN,
                      op(RowSrc::plain(sptr(st, L4D_STASH_CTX), nq), nq), Layout::MN, epi_acc(dw->o, nq), dwpart)))
      return r;
    // attention backward -> dQKV (inverse RoPE applied), remote dK/dV
    AttnParams ap = attn_params(x);
    ap.q = sptr(st, L4D_STASH_Q);
    ap.o = sptr(st, L4D_STASH_CTX);
    ap.lse = sptr<float>(st, L4D_STASH_LSE);
    ap.dout = dctx;
    ap.delta = delta;
    ap.dq = dqkv;
    ap.dq_ld = qc;
    ap.rope = rope;
    key_segments(x, ap, sptr(st, L4D_STASH_K), sptr(st, L4D_STASH_V), static_cast<const uint16_t*>(pi.remote_k),
                 static_cast<const uint16_t*>(pi.remote_v), dqkv, static_cast<uint16_t*>(d_remote_k),
                 static_cast<uint16_t*>(d_remote_v), static_cast<const uint16_t*>(pi.cp_peer_dk),
                 static_cast<const uint16_t*>(pi.cp_peer_dv));
    ap.total_keys = 0;
    for (int i = 0; i < ap.n_seg; ++i) {
      ap.seg_key0[i] = ap.total_keys;
      ap.total_keys += ap.seg[i].n;
    }
    ap.n_split = attn_bwd_splits(ap);
    if (ap.n_split > 1) {
      ap.dkv_partial = reinterpret_cast<float*>(wsb + plan.dkv);
      ap.partial_half = (int64_t)ap.n_split * x.b * ap.total_keys * x.k_t * x.d;
    }
    // dQ first: it also writes delta = rowsum(dO * O), which dK/dV reads
    if ((r = launch("attn_bwd_dq", s, [&] { return attn_bwd(ap, 2, s); }))) return r;
    if ((r = launch("attn_bwd_dkdv", s, [&] { return attn_bwd(ap, 1, s); }))) return r;
    if (ap.n_split > 1 && (r = launch("attn_dkv_reduce", s, [&] { return attn_bwd(ap, 3, s); }))) return r;
    // QKV projection
    if ((r = run_gemm("gemm_qkv_dx", s, tok, x.h, qc, op(RowSrc::plain(dqkv, qc), tok), Layout::KC,
                      op(RowSrc::plain(w->qkv, x.h), x.h), Layout::MN,
                      epi_residual(x, nullptr, nullptr, pi.sp_peer_dxn1, dxn1_send, dxn1))))
      return r;
    const RowSrc xn1_full = gathered(sptr(st, L4D_STASH_XN1), pi.sp_peer_xn1, x);
    if ((r = run_gemm("gemm_qkv_dw", s, qc, x.h, tok, op(RowSrc::plain(dqkv, qc), qc), Layout::MN, op(xn1_full, x.h),
                      Layout::MN, epi_acc(dw->qkv, x.h), dwpart)))
      return r;
    // norm-1 backward + residual
    if ((r = launch("rmsnorm1_bwd", s, [&] {
           const NormBwdIo io{nullptr, dxn1, nullptr, dh1_f32, static_cast<uint16_t*>(dx), nullptr};
           return rmsnorm_bwd(sptr(st, L4D_STASH_X), static_cast<const uint16_t*>(w->norm1), io, partial, npart,
                              rows_sp, (int32_t)x.h, x.eps, s);
         })))
      return r;
    if ((r = launch("reduce_gain", s, [&] { return reduce_rows_add(partial, npart, (int32_t)x.h, dw->norm1, s); })))
      return r;
    return L4D_OK;
  };
  rc = body();
  if (rc) return rc;
  return l4d_stash_release(A, st);
}

// ============================================================== LM head

namespace {
// Bytes of workspace the LM head needs: the bf16 logits, plus an fp32 n x h
// sum of d_hidden when the vocabulary shard has a ragged tail (ragged_k_split).
uint64_t lm_xent_ws_bytes(int64_t n, int64_t h, int64_t v_t) {
  return align_up((uint64_t)n * v_t * 2) + (ragged_k_split(v_t) ? align_up((uint64_t)n * h * 4) : 0);
}

int lm_xent_check(int64_t n, int64_t h, int64_t v_t, int64_t v0, const void* hidden, const void* w_lm,
                  const int64_t* targets, const float* peer_lse, const float* peer_z, const float* loss,
                  const void* d_hidden, const float* d_w) {
  if (n < 0 || h <= 0 || v_t <= 0 || v0 < 0) return fail(L4D_EINVAL, "bad LM-head sizes");
  if (h % 8 || v_t % 8) return fail(L4D_EINVAL, "hidden and vocab shard must be multiples of 8");
  if (n * v_t > ((int64_t)1 << 40) || n > INT32_MAX || v_t > INT32_MAX) return fail(L4D_EINVAL, "problem too large");
  if (!hidden || !w_lm || !targets || !loss || !d_hidden || !d_w)
    return fail(L4D_EINVAL, "hidden, w_lm, targets, loss, d_hidden and d_w_lm are required");
  if ((peer_lse == nullptr) != (peer_z == nullptr))
    return fail(L4D_EINVAL, "peer_lse and peer_target_logit go together");
  return L4D_OK;
}

// The LM-head kernel sequence over lm_xent_ws_bytes(n, h, v_t) bytes of
// device workspace at ws (256-byte aligned; nothing in it needs to start at
// zero: every byte is written before it is read).
int lm_xent_run(int64_t n, int64_t h, int64_t v_t, int64_t v0, const void* hidden, const void* w_lm,
                const int64_t* targets, const float* peer_lse, const float* peer_z, float grad_scale, float* loss,
                void* d_hidden, float* d_w, uint8_t* ws, hipStream_t s) {
  const uint64_t logit_bytes = align_up((uint64_t)n * v_t * 2);
  const bool split_k = ragged_k_split(v_t);
  uint16_t* logits = reinterpret_cast<uint16_t*>(ws);
  float* dh_f32 = split_k ? reinterpret_cast<float*>(ws + logit_bytes) : nullptr;
  int rc;
  if ((rc = run_gemm("gemm_lm_logits", s, n, v_t, h, op(RowSrc::plain(hidden, h), n), Layout::KC,
                     op(RowSrc::plain(w_lm, h), v_t), Layout::KC, epi_store(logits, v_t))))
    return rc;
  if ((rc = launch("xent_rows", s, [&] {
         return xent_rows(logits, n, (int32_t)v_t, v0, targets, peer_lse, peer_z, grad_scale, loss, logits, s);
       })))
    return rc;
  if (!split_k) {
    if ((rc = run_gemm("gemm_lm_dx", s, n, h, v_t, op(RowSrc::plain(logits, v_t), n), Layout::KC,
                       op(RowSrc::plain(w_lm, h), h), Layout::MN, epi_store(d_hidden, h))))
      return rc;
  } else {
    // d_hidden = dlogits[:, :K1] W_lm[:K1] + dlogits[:, K1:] W_lm[K1:] in fp32, then bf16
    const int64_t k1 = v_t - v_t % 128, k2 = v_t - k1;
    EpiParams ef{};
    ef.kind = EpiKind::StoreF32;
    ef.c = dh_f32;
    ef.ldc = h;
    if ((rc = run_gemm("gemm_lm_dx", s, n, h, k1, op(RowSrc::plain(logits, v_t), n), Layout::KC,
                       op(RowSrc::plain(w_lm, h), h), Layout::MN, ef)))
      return rc;
    if ((rc = run_gemm("gemm_lm_dx_tail", s, n, h, k2, op(RowSrc::plain(logits + k1, v_t), n), Layout::KC,
                       op(RowSrc::plain(static_cast<const uint16_t*>(w_lm) + k1 * h, h), h), Layout::MN,
                       epi_acc(dh_f32, h))))
      return rc;
    if ((rc = launch("gemm_splitk_reduce", s, [&] {
           return gemm_split_store(static_cast<uint16_t*>(d_hidden), h, dh_f32, n, h, 1, s);
         })))
      return rc;
  }
  return run_gemm("gemm_lm_dw", s, v_t, h, n, op(RowSrc::plain(logits, v_t), v_t), Layout::MN,
                  op(RowSrc::plain(hidden, h), h), Layout::MN, epi_acc(d_w, h));
}

// Workspace of lm_head_xent_noalloc: one array per device, held by the loaded
// code object until the process ends.  Host code must use the address that
// hipGetSymbolAddress returns for the current device, never the array's name.
constexpr uint64_t kScratchBytes = 64ull << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, resolved once per device.
int scratch_on_current_device(uint8_t** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(L4D_EDEVICE, "device %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(L4D_EDEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = static_cast<uint8_t*>(g_scratch_ptr[dev]);
  return L4D_OK;
}
}  // namespace

extern "C" int lm_head_xent(int64_t n, int64_t h, int64_t v_t, int64_t v0, const void* hidden, const void* w_lm,
                            const int64_t* targets, const float* peer_lse, const float* peer_z, float grad_scale,
                            float* loss, void* d_hidden, float* d_w, l4d_arena* A, void* stream_ptr) {
  int rc = lm_xent_check(n, h, v_t, v0, hidden, w_lm, targets, peer_lse, peer_z, loss, d_hidden, d_w);
  if (rc) return rc;
  if (!A) return fail(L4D_EINVAL, "arena is required");
  if (n == 0) return L4D_OK;
  Workspace ws;
  if ((rc = take_ws(A, lm_xent_ws_bytes(n, h, v_t), ws))) return rc;
  return lm_xent_run(n, h, v_t, v0, hidden, w_lm, targets, peer_lse, peer_z, grad_scale, loss, d_hidden, d_w,
                     reinterpret_cast<uint8_t*>(A->base + ws.off), static_cast<hipStream_t>(stream_ptr));
}

extern "C" int lm_head_xent_noalloc(int64_t n, int64_t h, int64_t v_t, int64_t v0, const void* hidden,
                                    const void* w_lm, const int64_t* targets, const float* peer_lse,
                                    const float* peer_z, float grad_scale, float* loss, void* d_hidden, float* d_w,
                                    void* stream_ptr) {
  int rc = lm_xent_check(n, h, v_t, v0, hidden, w_lm, targets, peer_lse, peer_z, loss, d_hidden, d_w);
  if (rc) return rc;
  const uint64_t need = lm_xent_ws_bytes(n, h, v_t);
  if (need > kScratchBytes)
    return fail(L4D_EINVAL, "LM head needs %llu bytes of workspace; the static scratch holds %llu",
                (unsigned long long)need, (unsigned long long)kScratchBytes);
  if (n == 0) return L4D_OK;
  uint8_t* ws = nullptr;
  if ((rc = scratch_on_current_device(&ws))) return rc;
  return lm_xent_run(n, h, v_t, v0, hidden, w_lm, targets, peer_lse, peer_z, grad_scale, loss, d_hidden, d_w, ws,
                     static_cast<hipStream_t>(stream_ptr));
}

// ============================================================== the ends of the model

namespace {
bool same_shard(const Shard& a, const Shard& b) {
  return a.h == b.h && a.a == b.a && a.k == b.k && a.f == b.f && a.s == b.s && a.b == b.b && a.t == b.t &&
         a.c == b.c && a.tr == b.tr && a.cr == b.cr;
}

int check_ends_stash(l4d_arena* A, const l4d_stash* st, int kind, const Shard& x) {
  if (!st || !A) return fail(L4D_EINVAL, "stash and arena are required");
  if (st->arena != A || !A->live.count(st)) return fail(L4D_EINVAL, "stash does not belong to this arena");
  if (st->kind != kind) return fail(L4D_EINVAL, kind == kHeadStash ? "not an LM-head stash" : "not an embedding stash");
  if (!same_shard(st->shape, x)) return fail(L4D_EINVAL, "stash was made for another shape");
  return L4D_OK;
}

// Vocabulary shard of this TP rank; v % t and (v/t) % 8 are required.
int vocab_shard(const l4d_model* m, const Shard& x, int64_t* v_t, int64_t* v0) {
  if (m->vocab % x.t) return fail(L4D_EINVAL, "vocab %% tp != 0");
  *v_t = m->vocab / x.t;
  if (*v_t % 8) return fail(L4D_EINVAL, "vocab / tp must be a multiple of 8");
  if ((int64_t)x.b * x.s_c * *v_t > ((int64_t)1 << 40)) return fail(L4D_EINVAL, "problem too large");
  *v0 = x.tr * *v_t;
  return L4D_OK;
}
}  // namespace

extern "C" int embedding_fwd(const l4d_model* m, const l4d_parallel* p, const int64_t* ids, const void* w_emb,
                             const void* receipt, void* send, void* x_out, l4d_arena* A, l4d_stash** stash_out,
                             void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  int64_t v_t, v0;
  if ((rc = vocab_shard(m, x, &v_t, &v0))) return rc;
  if (!ids || !w_emb || !x_out || !A || !stash_out) return fail(L4D_EINVAL, "ids, w_emb, x_out, arena and stash_out are required");
  if ((x.t > 1) != (send != nullptr)) return fail(L4D_EINVAL, "send is required iff tp > 1");
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);
  const uint64_t bytes[1] = {(uint64_t)x.b * x.s_c * 8};
  l4d_stash* st = nullptr;
  if ((rc = stash_reserve_sized(A, x, kEmbStash, L4D_EMB_COUNT, bytes, -1, &st))) return rc;
  auto body = [&]() -> int {
    HIP_TRY(hipMemcpyAsync(sptr<void>(st, L4D_EMB_IDS), ids, bytes[0], hipMemcpyDeviceToDevice, s));
    return launch("embed_fwd", s, [&] {
      return embed_fwd(ids, static_cast<const uint16_t*>(w_emb), v0, (int32_t)v_t, (int32_t)x.h, x.b * x.s_c,
                       (int32_t)x.s_c, (int32_t)x.s_sp, (int32_t)x.tr, (int32_t)x.t,
                       static_cast<const uint16_t*>(receipt), static_cast<uint16_t*>(x_out),
                       static_cast<uint16_t*>(send), s);
    });
  };
  if ((rc = body())) {
    l4d_stash_release(A, st);
    return rc;
  }
  *stash_out = st;
  return L4D_OK;
}

extern "C" int embedding_bwd(const l4d_model* m, const l4d_parallel* p, l4d_stash* st, const void* dx,
                             const void* peer_dx, float* d_w_emb, l4d_arena* A, void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  int64_t v_t, v0;
  if ((rc = vocab_shard(m, x, &v_t, &v0))) return rc;
  if ((rc = check_ends_stash(A, st, kEmbStash, x))) return rc;
  if (!dx || !d_w_emb) return fail(L4D_EINVAL, "dx and d_w_emb are required");
  if ((x.t > 1) != (peer_dx != nullptr)) return fail(L4D_EINVAL, "peer_dx is required iff tp > 1");
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);
  if ((rc = launch("embed_bwd", s, [&] {
         return embed_bwd(sptr<const int64_t>(st, L4D_EMB_IDS), gathered(dx, peer_dx, x), v0, (int32_t)v_t,
                          (int32_t)x.h, x.b * x.s_c, d_w_emb, s);
       })))
    return rc;
  return l4d_stash_release(A, st);
}

extern "C" int lm_head_fwd(const l4d_model* m, const l4d_parallel* p, const void* x_in, const void* w_norm,
                           const void* w_lm, const int64_t* targets, const void* peer_xn, const float* peer_lse,
                           const float* peer_z, float* loss, l4d_arena* A, l4d_stash** stash_out, void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  int64_t v_t, v0;
  if ((rc = vocab_shard(m, x, &v_t, &v0))) return rc;
  if (!x_in || !w_norm || !w_lm || !targets || !loss || !A || !stash_out)
    return fail(L4D_EINVAL, "x, w_norm, w_lm, targets, loss, arena and stash_out are required");
  if (x.t > 1 && (!peer_xn || !peer_lse || !peer_z))
    return fail(L4D_EINVAL, "tp > 1 needs peer_xn, peer_lse and peer_target_logit");
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);
  const int64_t tok = x.b * x.s_c;
  const uint64_t sp = (uint64_t)x.b * x.s_sp * x.h * 2;
  const uint64_t bytes[L4D_HEAD_COUNT] = {sp, sp, (uint64_t)tok * v_t * 4};
  l4d_stash* st = nullptr;
  if ((rc = stash_reserve_sized(A, x, kHeadStash, L4D_HEAD_COUNT, bytes, -1, &st))) return rc;
  auto body = [&]() -> int {
    int r;
    if ((r = launch("rmsnorm_fwd", s, [&] {
           return rmsnorm_fwd(static_cast<const uint16_t*>(x_in), static_cast<const uint16_t*>(w_norm),
                              sptr(st, L4D_HEAD_XN), x.b * x.s_sp, (int32_t)x.h, x.eps, s, sptr(st, L4D_HEAD_X));
         })))
      return r;
    EpiParams e{};
    e.kind = EpiKind::StoreF32;
    e.c = sptr<float>(st, L4D_HEAD_PROBS);
    e.ldc = v_t;
    if ((r = run_gemm("gemm_head_logits", s, tok, v_t, x.h, op(gathered(sptr(st, L4D_HEAD_XN), peer_xn, x), tok),
                      Layout::KC, op(RowSrc::plain(w_lm, x.h), v_t), Layout::KC, e)))
      return r;
    return launch("xent_probs", s, [&] {
      return xent_probs(sptr<float>(st, L4D_HEAD_PROBS), tok, (int32_t)v_t, v0, targets, peer_lse, peer_z, loss, s);
    });
  };
  if ((rc = body())) {
    l4d_stash_release(A, st);
    return rc;
  }
  *stash_out = st;
  return L4D_OK;
}

extern "C" int lm_head_bwd(const l4d_model* m, const l4d_parallel* p, const void* w_norm, const void* w_lm,
                           const int64_t* targets, const void* peer_xn, const void* peer_dxn, void* dxn_send,
                           float grad_scale, l4d_stash* st, void* dx, float* d_w_norm, float* d_w_lm, l4d_arena* A,
                           void* stream_ptr) {
  Shard x;
  int rc = make_shard(m, p, &x);
  if (rc) return rc;
  int64_t v_t, v0;
  if ((rc = vocab_shard(m, x, &v_t, &v0))) return rc;
  if ((rc = check_ends_stash(A, st, kHeadStash, x))) return rc;
  if (!w_norm || !w_lm || !targets || !dx || !d_w_norm || !d_w_lm)
    return fail(L4D_EINVAL, "w_norm, w_lm, targets, dx, d_w_norm and d_w_lm are required");
  if (x.t > 1 && !peer_xn) return fail(L4D_EINVAL, "tp > 1 needs peer_xn");
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);
  const int64_t tok = x.b * x.s_c, rows_sp = x.b * x.s_sp;
  const int32_t npart = rmsnorm_bwd_partials(rows_sp);
  Carver cv;
  const uint64_t o_dl = cv.take((uint64_t)tok * v_t * 2), o_dxn = cv.take((uint64_t)rows_sp * x.h * 2);
  const uint64_t o_part = cv.take((uint64_t)npart * x.h * 4);
  const uint64_t o_send = (x.t > 1 && !dxn_send) ? cv.take((uint64_t)x.b * (x.t - 1) * x.s_sp * x.h * 2) : 0;
  const bool split_k = ragged_k_split(v_t);
  const uint64_t o_sum = split_k ? cv.take((uint64_t)tok * x.h * 4) : 0;
  Workspace ws;
  if ((rc = take_ws(A, cv.used, ws))) return rc;
  uint8_t* wsb = reinterpret_cast<uint8_t*>(A->base + ws.off);
  uint16_t* dl = reinterpret_cast<uint16_t*>(wsb + o_dl);
  uint16_t* dxn = reinterpret_cast<uint16_t*>(wsb + o_dxn);
  float* partial = reinterpret_cast<float*>(wsb + o_part);
  void* send = x.t > 1 ? (dxn_send ? dxn_send : (void*)(wsb + o_send)) : nullptr;
  if ((rc = launch("xent_grad", s, [&] {
         return xent_grad(sptr<const float>(st, L4D_HEAD_PROBS), tok, (int32_t)v_t, v0, targets, grad_scale, dl, s);
       })))
    return rc;
  // d(xn) over the gathered rows: own rows + the peers' partials, the peers' rows sent
  if (!split_k) {
    if ((rc = run_gemm("gemm_head_dx", s, tok, x.h, v_t, op(RowSrc::plain(dl, v_t), tok), Layout::KC,
                       op(RowSrc::plain(w_lm, x.h), x.h), Layout::MN, epi_residual(x, dxn, nullptr, peer_dxn, send))))
      return rc;
  } else {   // as in lm_head_xent: the bulk of K on the BK = 64 kernel, the tail on the ragged one, in fp32
    float* sum = reinterpret_cast<float*>(wsb + o_sum);
    const int64_t k1 = v_t - v_t % 128, k2 = v_t - k1;
    EpiParams ef{};
    ef.kind = EpiKind::StoreF32;
    ef.c = sum;
    ef.ldc = x.h;
    if ((rc = run_gemm("gemm_head_dx", s, tok, x.h, k1, op(RowSrc::plain(dl, v_t), tok), Layout::KC,
                       op(RowSrc::plain(w_lm, x.h), x.h), Layout::MN, ef)))
      return rc;
    if ((rc = run_gemm("gemm_head_dx_tail", s, tok, x.h, k2, op(RowSrc::plain(dl + k1, v_t), tok), Layout::KC,
                       op(RowSrc::plain(static_cast<const uint16_t*>(w_lm) + k1 * x.h, x.h), x.h), Layout::MN,
                       epi_acc(sum, x.h))))
      return rc;
    if ((rc = launch("sp_finish", s, [&] {
           return sp_finish(sum, (int32_t)x.h, tok, (int32_t)x.s_c, (int32_t)x.s_sp, (int32_t)x.tr, (int32_t)x.t,
                            static_cast<const uint16_t*>(peer_dxn), dxn, static_cast<uint16_t*>(send), s);
         })))
      return rc;
  }
  if ((rc = launch("rmsnorm_bwd", s, [&] {
         const NormBwdIo io{dxn, nullptr, nullptr, nullptr, static_cast<uint16_t*>(dx), nullptr};
         return rmsnorm_bwd(sptr(st, L4D_HEAD_X), static_cast<const uint16_t*>(w_norm), io, partial, npart,
                            rows_sp, (int32_t)x.h, x.eps, s);
       })))
    return rc;
  if ((rc = launch("reduce_gain", s, [&] { return reduce_rows_add(partial, npart, (int32_t)x.h, d_w_norm, s); })))
    return rc;
  if ((rc = run_gemm("gemm_head_dw", s, v_t, x.h, tok, op(RowSrc::plain(dl, v_t), v_t), Layout::MN,
                     op(gathered(sptr(st, L4D_HEAD_XN), peer_xn, x), x.h), Layout::MN, epi_acc(d_w_lm, x.h))))
    return rc;
  return l4d_stash_release(A, st);
}

// ============================================================== optimizer

extern "C" int l4d_adam_step(const l4d_adam* hp, int64_t n, float* grad, float* master, float* m, float* v,
                             void* weight, void* stream_ptr) {
  if (!hp) return fail(L4D_EINVAL, "hyperparameters are required");
  if (n < 0) return fail(L4D_EINVAL, "n must be >= 0");
  if (hp->step < 1) return fail(L4D_EINVAL, "step counts from 1");
  if (!(hp->beta1 >= 0.f && hp->beta1 < 1.f) || !(hp->beta2 >= 0.f && hp->beta2 < 1.f))
    return fail(L4D_EINVAL, "beta1 and beta2 must lie in [0, 1)");
  if (!(hp->eps >= 0.f) || !std::isfinite(hp->eps)) return fail(L4D_EINVAL, "eps must be finite and >= 0");
  if (!std::isfinite(hp->lr) || !std::isfinite(hp->weight_decay) || !std::isfinite(hp->grad_scale))
    return fail(L4D_EINVAL, "lr, weight_decay and grad_scale must be finite");
  if (!grad || !master || !m || !v || !weight) return fail(L4D_EINVAL, "grad, master, m, v and weight are required");
  const void* f32s[4] = {grad, master, m, v};
  for (const void* p : f32s)
    if (reinterpret_cast<uintptr_t>(p) % 16) return fail(L4D_EINVAL, "fp32 arrays must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(weight) % 8) return fail(L4D_EINVAL, "the weight must be 8-byte aligned");
  if (n == 0) return L4D_OK;
  if (n > (int64_t(1) << 33)) return fail(L4D_EINVAL, "shard too large (more than 2^33 parameters)");
  const uintptr_t lo[5] = {(uintptr_t)grad, (uintptr_t)master, (uintptr_t)m, (uintptr_t)v, (uintptr_t)weight};
  const uint64_t len[5] = {4ull * n, 4ull * n, 4ull * n, 4ull * n, 2ull * n};
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (lo[i] < lo[j] + len[j] && lo[j] < lo[i] + len[i]) return fail(L4D_EINVAL, "the arrays overlap");
  const double b1 = hp->beta1, b2 = hp->beta2, t = static_cast<double>(hp->step);
  AdamConsts c;
  c.beta1 = hp->beta1;
  c.beta2 = hp->beta2;
  c.one_m_beta1 = static_cast<float>(1.0 - b1);
  c.one_m_beta2 = static_cast<float>(1.0 - b2);
  c.lr = hp->lr;
  c.decay = static_cast<float>(static_cast<double>(hp->lr) * hp->weight_decay);
  c.r1 = static_cast<float>(1.0 / -std::expm1(t * std::log(b1)));
  c.rs2 = static_cast<float>(1.0 / std::sqrt(-std::expm1(t * std::log(b2))));
  c.eps = hp->eps;
  c.scale = hp->grad_scale;
  c.scale_dev = hp->grad_scale_dev;
  hipStream_t s = static_cast<hipStream_t>(stream_ptr);
  return launch("adam_step", s, [&] {
    return adam_step(c, n, grad, master, m, v, static_cast<uint16_t*>(weight), hp->zero_grad, s);
  });
}
