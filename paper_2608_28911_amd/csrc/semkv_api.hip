// semkv_api.hip -- host side of the C ABI declared in include/semkv.h:
// validation, buffer geometry, host-side counts of the deferred state machine
// (Alg. 2) and kernel launches.  Nothing here allocates or synchronizes.
#include <math.h>
#include <string.h>

#include <array>
#include <map>
#include <mutex>

#include "semkv.h"
#include "semkv_internal.h"

using namespace semkv;

namespace {

// the adjacent pairs of the rest of the level grid (8/7, 7/6, 3/2 levels),
// for uniform sweeps (Sec. 4.2): per-row metadata only
bool grid_pair(int lh, int ll) { return (lh == 8 && ll == 7) || (lh == 7 && ll == 6) || (lh == 3 && ll == 2); }

bool levels_ok(int base, int lh, int ll) {
  if (base == SEMKV_BASE_TQ) return lh == 4 && ll == 3;
  if (grid_pair(lh, ll)) return true;
  if (base == SEMKV_BASE_ROT_AFFINE) return (lh == 6 && ll == 5) || (lh == 5 && ll == 4);
  static const int pairs[][2] = {{6, 5}, {5, 4}, {6, 4}, {4, 3}, {5, 3}, {6, 3}};
  for (auto& p : pairs)
    if (p[0] == lh && p[1] == ll) return true;
  return false;
}

int64_t top_count(int64_t T, int64_t rn, int64_t rd) { return rn * T / rd; }   // floor(r T)

int64_t round_half_even(int64_t n, int64_t rn, int64_t rd) {                    // round(r n)
  int64_t a = rn * n, q = a / rd, rem = a - q * rd;
  if (2 * rem > rd || (2 * rem == rd && (q & 1))) ++q;
  return q;
}

PoolGeom geom(const semkv_cache* c) {
  PoolGeom g;
  memset(&g, 0, sizeof(g));
  const semkv_config& k = c->cfg;
  g.pools = c->pools;
  g.unit_stride = c->sz.unit_stride;
  g.lo_offset = c->sz.cap_hi_tiles * c->sz.record_bytes_hi;
  g.rec_bytes[0] = int32_t(c->sz.record_bytes_hi);
  g.rec_bytes[1] = int32_t(c->sz.record_bytes_lo);
  g.tile_bytes[0] = int32_t(c->sz.tile_bytes_hi);
  g.tile_bytes[1] = int32_t(c->sz.tile_bytes_lo);
  g.meta_bytes = int32_t(c->sz.meta_bytes);
  g.L[0] = k.L_hi;
  g.L[1] = k.L_lo;
  g.base = k.base;
  g.G = k.group;
  g.n_layers = k.n_layers;
  g.n_kv_heads = k.n_kv_heads;
  g.batch = k.batch;
  memcpy(g.tau[0], c->tau_hi, sizeof(g.tau[0]));
  memcpy(g.tau[1], c->tau_lo, sizeof(g.tau[1]));
  g.signs = c->signs;
  g.status = c->status;
  return g;
}

bool all_appended(const semkv_cache* c) {
  for (int l = 0; l < c->cfg.n_layers; ++l)
    if (!((c->appended[l >> 5] >> (l & 31)) & 1u)) return false;
  return true;
}

bool none_appended(const semkv_cache* c) {
  return !(c->appended[0] | c->appended[1] | c->appended[2] | c->appended[3]);
}

// standard normal density and tail
double npdf(double x) { return exp(-0.5 * x * x) / sqrt(2.0 * M_PI); }
double ncdf(double x) { return 0.5 * erfc(-x / sqrt(2.0)); }

template <class F>
double bisect(F f, double lo, double hi) {
  double flo = f(lo);
  for (int it = 0; it < 200; ++it) {
    double mid = 0.5 * (lo + hi);
    if (mid == lo || mid == hi) break;
    double fm = f(mid);
    if ((fm < 0) == (flo < 0)) {
      lo = mid;
      flo = fm;
    } else {
      hi = mid;
    }
  }
  return 0.5 * (lo + hi);
}

// Workgroups the device holds at once for this cache's decode kernel (compute
// units x workgroups per unit), looked up once per device and level pair.
int64_t decode_slots(const semkv_config& k) {
  static std::mutex mu;
  static std::map<std::array<int, 5>, int64_t> known;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  const std::array<int, 5> key{dev, k.base, k.L_hi, k.L_lo, k.group};
  std::lock_guard<std::mutex> lock(mu);
  auto it = known.find(key);
  if (it != known.end()) return it->second;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 256;
  const int64_t slots = int64_t(cus) * decode_blocks_per_cu(k.base, k.L_hi, k.L_lo, k.group);
  known[key] = slots;
  return slots;
}

// Records on the busiest SIMD when a unit's nt tiles are dealt to ns
// workgroups of nw waves: slot s = wave * ns + split takes tiles s, s +
// stride, ... (stride = ns * nw), so slot s holds full + (s < left) tiles
// (full = nt div stride, left = nt mod stride); waves w and w + nw/2 share a
// SIMD, and the SIMD of split 0's waves 0 and nw/2 holds the most.
int64_t busiest_simd(int64_t nt, int64_t ns, int nw) {
  const int64_t stride = ns * nw, full = nt / stride, left = nt % stride;
  return 2 * full + (left > 0) + (left > ns * (nw / 2));
}

// Decode split plan: the tiles of each (sequence, kv head) unit, high pool
// then low pool, are dealt to nsplit workgroups (tile u to wave slot u mod
// nsplit * waves), at most as many workgroups as are resident at once: of
// those split counts, the one that leaves the busiest SIMD the fewest
// records, and of equals the largest (the most compute units at work; a short
// context then leaves some waves without a record rather than giving one
// SIMD a record more).  The fp16 tail rides with the last workgroup.  0:
// nothing cached.  A launch of `layers` layers plans over all their units
// together.
int plan(const semkv_cache* c, int n_tail, int layers = 1) {
  const int64_t nt = (c->n_hi + kSlots - 1) / kSlots + (c->n_lo + kSlots - 1) / kSlots;
  if (nt == 0) return n_tail > 0 ? 1 : 0;
  const int64_t units = int64_t(c->cfg.batch) * c->cfg.n_kv_heads * layers;
  int64_t ns_max = decode_slots(c->cfg) / units;
  const int nw = decode_waves(c->cfg.base, c->cfg.L_hi, c->cfg.L_lo, c->cfg.group);
  if (ns_max > nt) ns_max = nt;                  // every workgroup holds a tile
  if (ns_max > kMaxSplits / layers) ns_max = kMaxSplits / layers;
  if (ns_max < 1) ns_max = 1;
  int64_t best = ns_max, best_load = busiest_simd(nt, ns_max, nw);
  for (int64_t ns = ns_max - 1; ns >= 1; --ns) {
    const int64_t load = busiest_simd(nt, ns, nw);
    if (load < best_load) {
      best = ns;
      best_load = load;
    }
  }
  return int(best);
}

// workspace: [layer][b][kvh] uint32 counters, one per 256-byte line, then the
// partials.  The counter prefix is sized for every layer whatever the launch:
// a one-layer launch uses its first batch x kv-head counters, an all-layers
// launch all of them, and the partials of either kind start past the whole
// prefix, so no launch writes partials where another kind keeps counters.
size_t counter_bytes(const semkv_config& k) {
  return size_t(int64_t(k.n_layers) * k.batch * k.n_kv_heads * kCounterStride * 4);
}

size_t workspace_need(const semkv_config& k, int nsplit, int layers) {
  return counter_bytes(k) + size_t(int64_t(layers) * k.batch * k.n_kv_heads * nsplit * 4 * kPartial * 4);
}

int close_block(semkv_cache* c, int n, hipStream_t stream) {
  const semkv_config& k = c->cfg;
  int64_t kh = round_half_even(n, k.r_num, k.r_den);
  if (c->n_hi + kh > c->sz.cap_hi_tiles * kSlots || c->n_lo + (n - kh) > c->sz.cap_lo_tiles * kSlots)
    return SEMKV_ECAPACITY;
  int64_t pos0 = c->n_hi + c->n_lo;
  if (pos0 + n > c->sz.flag_words * 32) return SEMKV_ECAPACITY;
  CloseArgs a;
  memset(&a, 0, sizeof(a));
  a.g = geom(c);
  a.tail = c->tail;
  a.tail_scores = c->tail_scores;
  a.n = n;
  a.k_hi = int32_t(kh);
  a.n0[0] = c->n_hi;
  a.n0[1] = c->n_lo;
  a.flags = c->flags;
  a.flag_words = c->sz.flag_words;
  a.pos0 = pos0;
  int st = launch_close(a, stream);
  if (st) return st;
  c->n_hi += kh;
  c->n_lo += n - kh;
  c->n_scored = 0;
  return SEMKV_OK;
}

__global__ void store_score_kernel(float* dst, const float* src, int slot, int batch) {
  int b = threadIdx.x;
  if (b < batch) dst[b * kSlots + slot] = src[b];
}

// zero n words (a kernel, not a memset node, so that a captured graph replays it)
__global__ void zero_words_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

// ---- scratch of semkv_decode_attn_noalloc ----------------------------
// A file-scope device array holds that entry point's finished-split counters
// (the first kScratchCounterBytes) and its split partials (the rest), so the
// call needs no workspace and allocates nothing.  Each GPU the library runs
// on holds its own copy until the process ends; every call on a GPU shares
// it.  The counters start at zero (cleared once per device by the set-up
// below) and every call leaves them zero; the partials are written before
// they are read.  In host code `scratch` names a host-side stand-in, never
// the device memory: the device address comes from hipGetSymbolAddress.
constexpr size_t kScratchBytes = size_t(8) << 20;
constexpr size_t kScratchCounterBytes = size_t(1) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// Device address of `scratch` on the current device.  The first call on a
// device looks it up and clears its counters with a fill kernel on `stream`
// (a kernel, not a memset node, so that a captured graph replays it).
int scratch_address(hipStream_t stream, uint8_t** out) {
  static std::mutex mu;
  static std::map<int, uint8_t*> known;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SEMKV_EHIP;
  std::lock_guard<std::mutex> lock(mu);
  auto it = known.find(dev);
  if (it == known.end()) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return SEMKV_EHIP;
    const int64_t words = int64_t(kScratchCounterBytes / 4);
    hipLaunchKernelGGL(zero_words_kernel, dim3(unsigned((words + 255) / 256)), dim3(256), 0, stream,
                       static_cast<uint32_t*>(p), words);
    if (hipGetLastError() != hipSuccess) return SEMKV_EHIP;
    it = known.emplace(dev, static_cast<uint8_t*>(p)).first;
  }
  *out = it->second;
  return SEMKV_OK;
}

}  // namespace

extern "C" {

const char* semkv_strerror(int status) {
  switch (status) {
    case SEMKV_OK: return "ok";
    case SEMKV_EINVAL: return "invalid argument";
    case SEMKV_EUNSUPPORTED: return "unsupported configuration";
    case SEMKV_ECAPACITY: return "capacity exceeded";
    case SEMKV_ENAN: return "non-finite data";
    case SEMKV_EHIP: return "HIP runtime error";
    case SEMKV_ESTATE: return "call out of order";
    default: return "unknown status";
  }
}

int semkv_cache_sizes(const semkv_config* cfg, semkv_sizes* out) {
  if (!cfg || !out) return SEMKV_EINVAL;
  const semkv_config& k = *cfg;
  if (k.n_layers < 1 || k.n_kv_heads < 1 || k.batch < 1 || k.n_layers > 128) return SEMKV_EINVAL;
  if (k.r_den <= 0 || k.r_num < 0 || k.r_num > k.r_den || k.max_prompt < 0 || k.max_new < 0)
    return SEMKV_EINVAL;
  if (k.max_prompt + k.max_new > (int64_t(1) << 29)) return SEMKV_EINVAL;   // decode splits use 32-bit tile math
  // launch grids put (sequence x layer) and (kv head x pool) in dimensions of at most 65535
  if (int64_t(k.batch) * k.n_layers > 65535 || k.n_kv_heads > 4096) return SEMKV_EUNSUPPORTED;
  if (k.head_dim != 128 || k.n_q_heads != 4 * k.n_kv_heads || k.block != 64) return SEMKV_EUNSUPPORTED;
  if (k.base != SEMKV_BASE_AFFINE && k.base != SEMKV_BASE_TQ && k.base != SEMKV_BASE_ROT_AFFINE)
    return SEMKV_EUNSUPPORTED;
  if (!levels_ok(k.base, k.L_hi, k.L_lo)) return SEMKV_EUNSUPPORTED;
  if (k.base != SEMKV_BASE_TQ && k.group != 32 && k.group != 64 && k.group != 128) return SEMKV_EUNSUPPORTED;
  if (k.base == SEMKV_BASE_TQ && k.group != 128) return SEMKV_EUNSUPPORTED;
  if (grid_pair(k.L_hi, k.L_lo) && k.group != 128) return SEMKV_EUNSUPPORTED;
  // the decode kernel needs one 8-wave workgroup's tables and buffers in a
  // compute unit's LDS (6 and 3 levels with 32-channel groups do not fit)
  if (decode_waves(k.base, k.L_hi, k.L_lo, k.group) < 8) return SEMKV_EUNSUPPORTED;
  memset(out, 0, sizeof(*out));
  int64_t khi = top_count(k.max_prompt, k.r_num, k.r_den);
  int64_t hi_rows = khi + k.max_new, lo_rows = k.max_prompt - khi + k.max_new;
  out->cap_hi_tiles = (hi_rows + kSlots - 1) / kSlots;
  out->cap_lo_tiles = (lo_rows + kSlots - 1) / kSlots;
  if (out->cap_hi_tiles < 1) out->cap_hi_tiles = 1;
  if (out->cap_lo_tiles < 1) out->cap_lo_tiles = 1;
  out->tile_bytes_hi = tile_bytes(k.L_hi);
  out->tile_bytes_lo = tile_bytes(k.L_lo);
  out->meta_bytes = meta_bytes(k.base, k.group);
  out->record_bytes_hi = record_bytes(k.base, k.L_hi, k.group);
  out->record_bytes_lo = record_bytes(k.base, k.L_lo, k.group);
  out->unit_stride = out->cap_hi_tiles * out->record_bytes_hi + out->cap_lo_tiles * out->record_bytes_lo;
  int64_t units = int64_t(k.batch) * k.n_layers * k.n_kv_heads;
  out->pool_bytes = size_t(units * out->unit_stride);
  out->tail_bytes = size_t(units * 2 * kSlots * kD * 2);
  out->tail_score_bytes = size_t(k.batch) * kSlots * 4;
  out->flag_words = (k.max_prompt + k.max_new + 31) / 32 + 1;
  out->flag_bytes = size_t(rank_scratch_offset(k.batch, out->flag_words) + k.batch * rank_scratch_words(k.max_prompt)) * 4;
  int64_t max_split = out->cap_hi_tiles + out->cap_lo_tiles;
  if (max_split > kMaxSplits) max_split = kMaxSplits;
  int64_t max_split_all = kMaxSplits / k.n_layers < 1 ? 1 : kMaxSplits / k.n_layers;   // all-layers launch
  if (max_split_all > max_split) max_split_all = max_split;
  const size_t one = workspace_need(k, int(max_split), 1), all = workspace_need(k, int(max_split_all), k.n_layers);
  out->workspace_bytes = one > all ? one : all;
  return SEMKV_OK;
}

int semkv_tq_codebook(int L, float* mu, float* tau) {
  if (!mu || !tau) return SEMKV_EINVAL;
  if (L == 2) {                      // cells (-inf, 0], (0, inf): centroid 2 phi(0)
    double m = 2.0 * npdf(0.0);
    mu[0] = float(-m);
    mu[1] = float(m);
    tau[0] = 0.0f;
    return SEMKV_OK;
  }
  if (L == 3) {                      // levels -m, 0, m; thresholds -m/2, m/2
    auto f = [](double m) { double t = 0.5 * m; return npdf(t) / (1.0 - ncdf(t)) - m; };
    double m = bisect(f, 0.5, 3.0);
    mu[0] = float(-m);
    mu[1] = 0.0f;
    mu[2] = float(m);
    tau[0] = float(-0.5 * m);
    tau[1] = float(0.5 * m);
    return SEMKV_OK;
  }
  if (L == 4) {                      // levels -b, -a, a, b; thresholds -t, 0, t with t = (a+b)/2
    auto inner = [](double t) { return (npdf(0.0) - npdf(t)) / (ncdf(t) - 0.5); };
    auto outer = [](double t) { return npdf(t) / (1.0 - ncdf(t)); };
    auto f = [&](double t) { return 0.5 * (inner(t) + outer(t)) - t; };
    double t = bisect(f, 0.1, 3.0);
    double a = inner(t), b = outer(t);
    mu[0] = float(-b);
    mu[1] = float(-a);
    mu[2] = float(a);
    mu[3] = float(b);
    tau[0] = float(-t);
    tau[1] = 0.0f;
    tau[2] = float(t);
    return SEMKV_OK;
  }
  return SEMKV_EUNSUPPORTED;
}

int semkv_cache_init(semkv_cache* c, const semkv_config* cfg, void* pools, void* tail,
                     float* tail_scores, uint32_t* flags, const uint32_t* signs, int32_t* status) {
  if (!c || !cfg) return SEMKV_EINVAL;
  semkv_sizes sz;
  int st = semkv_cache_sizes(cfg, &sz);
  if (st) return st;
  if (!pools || !tail || !tail_scores || !flags || !status) return SEMKV_EINVAL;
  if (cfg->base != SEMKV_BASE_AFFINE && !signs) return SEMKV_EINVAL;
  if ((uintptr_t(pools) | uintptr_t(tail)) & 15) return SEMKV_EINVAL;
  memset(c, 0, sizeof(*c));
  c->cfg = *cfg;
  c->sz = sz;
  c->pools = static_cast<uint8_t*>(pools);
  c->tail = static_cast<uint16_t*>(tail);
  c->tail_scores = tail_scores;
  c->flags = flags;
  c->signs = signs;
  c->status = status;
  if (cfg->base == SEMKV_BASE_TQ) {
    semkv_tq_codebook(cfg->L_hi, c->mu_hi, c->tau_hi);
    semkv_tq_codebook(cfg->L_lo, c->mu_lo, c->tau_lo);
  }
  return SEMKV_OK;
}

int semkv_rank_sizes(const semkv_cache* c, int64_t T, int64_t* n_hi, int64_t* n_lo) {
  if (!c || !n_hi || !n_lo || T < 1) return SEMKV_EINVAL;
  if (T > c->cfg.max_prompt) return SEMKV_ECAPACITY;
  *n_hi = top_count(T, c->cfg.r_num, c->cfg.r_den);
  *n_lo = T - *n_hi;
  return SEMKV_OK;
}

int semkv_rank(semkv_cache* c, const float* scores, int64_t T, int32_t* hi_idx, int32_t* lo_idx,
               hipStream_t stream) {
  if (!c || !scores || T < 1) return SEMKV_EINVAL;
  if (T > c->cfg.max_prompt) return SEMKV_ECAPACITY;
  const int64_t kh = top_count(T, c->cfg.r_num, c->cfg.r_den);
  if ((kh > 0 && !hi_idx) || (kh < T && !lo_idx)) return SEMKV_EINVAL;   // an empty list may be NULL
  RankArgs a;
  a.scores = scores;
  a.T = T;
  a.K = top_count(T, c->cfg.r_num, c->cfg.r_den);
  a.ld_s = T;
  a.flags = c->flags;
  a.flag_words = c->sz.flag_words;
  a.hi_idx = hi_idx;
  a.lo_idx = lo_idx;
  a.status = c->status;
  a.scratch = c->flags + rank_scratch_offset(c->cfg.batch, c->sz.flag_words);
  a.scratch_words = rank_scratch_words(c->cfg.max_prompt);
  return launch_rank(a, c->cfg.batch, stream);
}

int semkv_quantize_pack(semkv_cache* c, int32_t layer, const uint16_t* K, const uint16_t* V,
                        int64_t sL, int64_t sB, int64_t sH, int64_t sT, int64_t T,
                        const int32_t* hi_idx, const int32_t* lo_idx, hipStream_t stream) {
  if (!c || !K || !V || T < 1) return SEMKV_EINVAL;
  const semkv_config& k = c->cfg;
  if (layer < -1 || layer >= k.n_layers) return SEMKV_EINVAL;
  if (T > k.max_prompt) return SEMKV_ECAPACITY;
  if (((uintptr_t(K) | uintptr_t(V)) & 15) || ((sB | sH | sT | (layer < 0 ? sL : 0)) & 7) || sT < 128)
    return SEMKV_EINVAL;
  int64_t kh = top_count(T, k.r_num, k.r_den);
  if ((kh > 0 && !hi_idx) || (kh < T && !lo_idx)) return SEMKV_EINVAL;
  bool fresh = c->n_hi == 0 && c->n_lo == 0 && c->n_prompt == 0;
  bool same = c->n_prompt == T && c->n_hi == kh && c->n_lo == T - kh;
  if (!fresh && !same) return SEMKV_ESTATE;   // generated blocks already closed
  QuantArgs a;
  memset(&a, 0, sizeof(a));
  a.g = geom(c);
  a.K = K;
  a.V = V;
  a.sL = sL;
  a.sB = sB;
  a.sH = sH;
  a.sT = sT;
  a.layer0 = layer < 0 ? 0 : layer;
  a.n_layers_launched = layer < 0 ? k.n_layers : 1;
  a.idx[0] = hi_idx;
  a.idx[1] = lo_idx;
  a.n_pool[0] = kh;
  a.n_pool[1] = T - kh;
  a.T = T;
  int64_t mt = ((kh > T - kh ? kh : T - kh) + kSlots - 1) / kSlots;
  a.max_tiles = int32_t(mt);
  int st = launch_quantize(a, stream);
  if (st) return st;
  c->n_prompt = T;
  c->n_hi = kh;
  c->n_lo = T - kh;
  return SEMKV_OK;
}

int semkv_append_kv(semkv_cache* c, int32_t layer, const uint16_t* k_new, const uint16_t* v_new,
                    hipStream_t stream) {
  if (!c || !k_new || !v_new) return SEMKV_EINVAL;
  const semkv_config& k = c->cfg;
  if (layer < -1 || layer >= k.n_layers) return SEMKV_EINVAL;
  if (c->n_hi + c->n_lo + c->n_scored + 1 > k.max_prompt + k.max_new) return SEMKV_ECAPACITY;
  if (c->n_scored >= kSlots) return SEMKV_ESTATE;
  if ((uintptr_t(k_new) | uintptr_t(v_new)) & 3) return SEMKV_EINVAL;
  AppendArgs a;
  a.tail = c->tail;
  a.k = k_new;
  a.v = v_new;
  a.layer0 = layer < 0 ? 0 : layer;
  a.n_layers_launched = layer < 0 ? k.n_layers : 1;
  a.n_layers = k.n_layers;
  a.n_kv_heads = k.n_kv_heads;
  a.batch = k.batch;
  a.slot = c->n_scored;
  int st = launch_append(a, stream);
  if (st) return st;
  for (int l = a.layer0; l < a.layer0 + a.n_layers_launched; ++l) c->appended[l >> 5] |= 1u << (l & 31);
  return SEMKV_OK;
}

int semkv_append_commit(semkv_cache* c, const float* score_new, hipStream_t stream) {
  if (!c || !score_new) return SEMKV_EINVAL;
  if (!all_appended(c)) return SEMKV_ESTATE;
  if (c->cfg.batch > 1024) return SEMKV_EUNSUPPORTED;
  hipLaunchKernelGGL(store_score_kernel, dim3(1), dim3(1024), 0, stream, c->tail_scores, score_new,
                     c->n_scored, c->cfg.batch);
  if (hipGetLastError() != hipSuccess) return SEMKV_EHIP;
  c->n_scored += 1;
  memset(c->appended, 0, sizeof(c->appended));
  if (c->n_scored == kSlots) return close_block(c, kSlots, stream);
  return SEMKV_OK;
}

int semkv_cache_reset(semkv_cache* c, hipStream_t stream) {
  if (!c || !c->flags) return SEMKV_EINVAL;
  const int64_t n = int64_t(c->cfg.batch) * c->sz.flag_words;
  const int64_t blocks = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
  hipLaunchKernelGGL(zero_words_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, c->flags, n);
  if (hipGetLastError() != hipSuccess) return SEMKV_EHIP;
  c->n_prompt = 0;
  c->n_hi = 0;
  c->n_lo = 0;
  c->n_scored = 0;
  memset(c->appended, 0, sizeof(c->appended));
  return SEMKV_OK;
}

int semkv_flush(semkv_cache* c, hipStream_t stream) {
  if (!c) return SEMKV_EINVAL;
  if (!none_appended(c)) return SEMKV_ESTATE;
  if (c->n_scored == 0) return SEMKV_OK;
  return close_block(c, c->n_scored, stream);
}

int semkv_workspace_bytes(const semkv_cache* c, size_t* bytes) {
  if (!c || !bytes) return SEMKV_EINVAL;
  const size_t one = workspace_need(c->cfg, plan(c, 1), 1);
  const size_t all = workspace_need(c->cfg, plan(c, 1, c->cfg.n_layers), c->cfg.n_layers);
  *bytes = one > all ? one : all;
  return SEMKV_OK;
}

// Decode launch of one layer; with k_new/v_new, the launch also stores them
// as the layer's current tail row (the fused append).
// Where a decode launch keeps its finished-split counters and its split
// partials: the caller's workspace, or the library's scratch array.
struct DecodeScratch {
  uint32_t* counters;       // [layer][b][kvh], zero between calls
  size_t counter_bytes;     // bytes available for them
  float* partials;          // split partials
  size_t partial_bytes;     // bytes available for them
};

// Decode launch of one layer; with k_new/v_new, the launch also stores them
// as the layer's current tail row (the fused append).  `too_small` is the
// status returned when the plan's counters or partials do not fit `sc`.
static int decode_launch(const semkv_cache* c, int32_t layer, int layers, int n_tail, const uint16_t* k_new,
                         const uint16_t* v_new, const uint16_t* q, float* out, const DecodeScratch& sc,
                         int too_small, hipStream_t stream) {
  const semkv_config& k = c->cfg;
  DecodeArgs a;
  memset(&a, 0, sizeof(a));
  const int nsplit = plan(c, n_tail, layers);
  if (nsplit == 0) return SEMKV_ESTATE;      // nothing cached yet
  if (sc.counter_bytes < counter_bytes(k) ||
      sc.partial_bytes < workspace_need(k, nsplit, layers) - counter_bytes(k))
    return too_small;
  a.g = geom(c);
  a.tail = c->tail;
  a.k_new = k_new;
  a.v_new = v_new;
  a.q = q;
  a.counters = sc.counters;
  a.ws = sc.partials;
  a.out = out;
  a.layer = layer;
  a.n_layers_launched = layers;
  a.n_rows[0] = c->n_hi;
  a.n_rows[1] = c->n_lo;
  a.n_tail = n_tail;
  a.nsplit = nsplit;
  memcpy(a.mu[0], c->mu_hi, sizeof(a.mu[0]));
  memcpy(a.mu[1], c->mu_lo, sizeof(a.mu[1]));
  return launch_decode(a, stream);
}

// the caller's workspace: counters for every layer, then the partials
static DecodeScratch workspace_scratch(const semkv_config& k, void* workspace, size_t ws_bytes) {
  const size_t cb = counter_bytes(k);
  DecodeScratch sc;
  sc.counters = static_cast<uint32_t*>(workspace);
  sc.counter_bytes = ws_bytes < cb ? ws_bytes : cb;
  sc.partials = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) + cb);
  sc.partial_bytes = ws_bytes > cb ? ws_bytes - cb : 0;
  return sc;
}

int semkv_decode_attn(const semkv_cache* c, int32_t layer, const uint16_t* q, float* out,
                      void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (!c || !q || !out || !workspace) return SEMKV_EINVAL;
  const semkv_config& k = c->cfg;
  if (layer < -1 || layer >= k.n_layers) return SEMKV_EINVAL;
  if ((uintptr_t(q) & 3) || (uintptr_t(workspace) & 15)) return SEMKV_EINVAL;
  if (layer == -1) {                         // every layer in one launch: one tail length for all
    const bool all = all_appended(c), none = none_appended(c);
    if (!all && !none) return SEMKV_ESTATE;
    return decode_launch(c, 0, k.n_layers, c->n_scored + (all ? 1 : 0), nullptr, nullptr, q, out,
                         workspace_scratch(k, workspace, ws_bytes), SEMKV_EINVAL, stream);
  }
  const int n_tail = c->n_scored + (((c->appended[layer >> 5] >> (layer & 31)) & 1u) ? 1 : 0);
  return decode_launch(c, layer, 1, n_tail, nullptr, nullptr, q, out, workspace_scratch(k, workspace, ws_bytes),
                       SEMKV_EINVAL, stream);
}

int semkv_decode_attn_noalloc(const semkv_cache* c, int32_t layer, const uint16_t* q, float* out,
                              hipStream_t stream) {
  if (!c || !q || !out) return SEMKV_EINVAL;
  const semkv_config& k = c->cfg;
  if (layer < -1 || layer >= k.n_layers) return SEMKV_EINVAL;
  if (uintptr_t(q) & 3) return SEMKV_EINVAL;
  // checks that need no device work come before the set-up
  const bool all = all_appended(c), none = none_appended(c);
  if (layer == -1 && !all && !none) return SEMKV_ESTATE;
  const int n_tail = layer == -1 ? c->n_scored + (all ? 1 : 0)
                                 : c->n_scored + (((c->appended[layer >> 5] >> (layer & 31)) & 1u) ? 1 : 0);
  if (plan(c, n_tail, layer == -1 ? k.n_layers : 1) == 0) return SEMKV_ESTATE;
  uint8_t* base = nullptr;
  const int st = scratch_address(stream, &base);
  if (st) return st;
  DecodeScratch sc;
  sc.counters = reinterpret_cast<uint32_t*>(base);
  sc.counter_bytes = kScratchCounterBytes;
  sc.partials = reinterpret_cast<float*>(base + kScratchCounterBytes);
  sc.partial_bytes = kScratchBytes - kScratchCounterBytes;
  if (layer == -1) return decode_launch(c, 0, k.n_layers, n_tail, nullptr, nullptr, q, out, sc, SEMKV_ECAPACITY, stream);
  return decode_launch(c, layer, 1, n_tail, nullptr, nullptr, q, out, sc, SEMKV_ECAPACITY, stream);
}

int semkv_append_decode(semkv_cache* c, int32_t layer, const uint16_t* k_new, const uint16_t* v_new,
                        const uint16_t* q, float* out, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (!c || !k_new || !v_new || !q || !out || !workspace) return SEMKV_EINVAL;
  const semkv_config& k = c->cfg;
  if (layer < 0 || layer >= k.n_layers) return SEMKV_EINVAL;
  if ((uintptr_t(k_new) | uintptr_t(v_new) | uintptr_t(q)) & 3 || (uintptr_t(workspace) & 15)) return SEMKV_EINVAL;
  if (((c->appended[layer >> 5] >> (layer & 31)) & 1u) != 0) return SEMKV_ESTATE;   // appended already
  if (c->n_hi + c->n_lo + c->n_scored + 1 > k.max_prompt + k.max_new) return SEMKV_ECAPACITY;
  if (c->n_scored >= kSlots) return SEMKV_ESTATE;
  const int st = decode_launch(c, layer, 1, c->n_scored + 1, k_new, v_new, q, out,
                               workspace_scratch(k, workspace, ws_bytes), SEMKV_EINVAL, stream);
  if (st) return st;
  c->appended[layer >> 5] |= 1u << (layer & 31);
  return SEMKV_OK;
}

int semkv_dequant(const semkv_cache* c, int32_t layer, float* k_hat, float* v_hat, hipStream_t stream) {
  if (!c || !k_hat || !v_hat) return SEMKV_EINVAL;
  if (layer < 0 || layer >= c->cfg.n_layers) return SEMKV_EINVAL;
  if ((uintptr_t(k_hat) | uintptr_t(v_hat)) & 15) return SEMKV_EINVAL;
  if (c->n_hi + c->n_lo == 0) return SEMKV_OK;
  DequantArgs a;
  memset(&a, 0, sizeof(a));
  a.g = geom(c);
  a.layer = layer;
  a.n_rows[0] = c->n_hi;
  a.n_rows[1] = c->n_lo;
  memcpy(a.mu[0], c->mu_hi, sizeof(a.mu[0]));
  memcpy(a.mu[1], c->mu_lo, sizeof(a.mu[1]));
  a.k_hat = k_hat;
  a.v_hat = v_hat;
  return launch_dequant(a, stream);
}

int semkv_score_hidden(int32_t indicator, const void* hidden, int32_t dtype, int32_t m, int32_t batch,
                       int64_t T, int32_t d_model, int64_t s_state, int64_t s_batch, int64_t s_token,
                       float* scores, hipStream_t stream) {
  if (!hidden || !scores || batch < 1 || T < 1 || m < 0) return SEMKV_EINVAL;
  if (indicator < SEMKV_IND_DELTA_NORM || indicator > SEMKV_IND_COSINE_DELTA) return SEMKV_EINVAL;
  if (dtype != SEMKV_DTYPE_F16 && dtype != SEMKV_DTYPE_BF16) return SEMKV_EINVAL;
  if ((indicator == SEMKV_IND_DELTA_NORM || indicator == SEMKV_IND_COSINE_DELTA) && m < 1) return SEMKV_EINVAL;
  if (d_model < 8 || d_model % 8) return SEMKV_EINVAL;
  if (d_model > 8192) return SEMKV_EUNSUPPORTED;
  if ((int64_t(batch) * T + 3) / 4 > int64_t(INT32_MAX)) return SEMKV_EUNSUPPORTED;   // one wave per token
  if ((uintptr_t(hidden) & 15) || (uintptr_t(scores) & 3) || ((s_state | s_batch | s_token) & 7)) return SEMKV_EINVAL;
  HiddenArgs a;
  a.h = static_cast<const uint16_t*>(hidden);
  a.s_state = s_state;
  a.s_batch = s_batch;
  a.s_token = s_token;
  a.indicator = indicator;
  a.dtype = dtype;
  a.m = m;
  a.batch = batch;
  a.d = d_model;
  a.T = T;
  a.scores = scores;
  return launch_score_hidden(a, stream);
}

int semkv_score_kv_norm(const semkv_cache* c, const uint16_t* X, int64_t sL, int64_t sB, int64_t sH,
                        int64_t sT, int64_t T, float* scores, hipStream_t stream) {
  if (!c || !X || !scores || T < 1) return SEMKV_EINVAL;
  if ((uintptr_t(X) & 15) || (uintptr_t(scores) & 3) || ((sL | sB | sH | sT) & 7) || sT < 128) return SEMKV_EINVAL;
  KvNormArgs a;
  a.X = X;
  a.sL = sL;
  a.sB = sB;
  a.sH = sH;
  a.sT = sT;
  a.n_layers = c->cfg.n_layers;
  a.n_kv_heads = c->cfg.n_kv_heads;
  a.batch = c->cfg.batch;
  a.T = T;
  a.scores = scores;
  return launch_kv_norm(a, stream);
}

}  // extern "C"
