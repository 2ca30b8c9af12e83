// C ABI of libhs2.so: argument checks, work planning, workspace layout and the
// launch sequence of each call.  Declarations and contracts: include/hs2.h.
#include "../../include/hs2.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "hs2_device.h"
#include "hs2_launch.h"

namespace {

using namespace hs2;

constexpr int kMaxQueries = 16;
constexpr int kMaxRows = 128;           // C * Gp
constexpr int kMaxGroup = 64;
constexpr int64_t kMaxGridRows = 65535;  // largest grid y extent: the (b, g, c) rows
constexpr int64_t kMaxTokenStride = 1 << 24;  // elements: 64 token rows stay below 2^31 bytes
constexpr int32_t kMaxLen = 1 << 27;
constexpr int kNBins = 1024;          // must match the kernels' first-level radix bins
constexpr int kSelChunk = hs2::SEL_CHUNK;  // tokens per workgroup of the selection scans
constexpr size_t kAlign = 256;
// share of each full-attention token group whose K rows stay cacheable when
// the score pass re-reads K (percent; the rest streams past the caches):
// the last half of each group's part of the split
constexpr int kFaKeepPercent = 50;
constexpr int64_t kLastLevelCacheBytes = 256ll << 20;  // MI355X memory-side cache

thread_local std::string g_last_error;

hs2_status fail(hs2_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}
int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

int env_int(const char* name, int dflt) {
  const char* v = getenv(name);
  if (!v || !*v) return dflt;
  return atoi(v);
}

// ---------------------------------------------------------------- planning
struct Plan {
  int B, C, Hq, Hkv, G, Gp, D, Lmax, k, W, S;
  float c2;
  int RT, TG;                 // full-attention / pooling row tiles
  int fa_variant;             // ring kernel shape (0, 2, 3, 4) for RT <= 4; 1: workgroup kernel
  FaSplitPlan fa_sp;          // full-attention token splits (grid: fa_sp.n_items items)
  int fa_cache_policy;  // FaCachePolicy of the full-attention ring kernel
  int fa_k_keep;        // FA_STREAM_K_HEAD: percent of each token group's K rows kept cacheable
  int logit_chunk;
  int pool_split, pool_nsplit;
  int64_t units;              // B * Hkv
  int64_t rows;               // selection rows B * Hkv * C
  int64_t score_stride, bitmap_words, cand_cap;
  int sel_nchunks;
  bool kv8;                   // E4M3 cache
  bool pool_logits;           // scores from logits stored by the full-attention kernel
  int64_t logit_stride;
  // workspace layout of hs2_full_attn_score_select / hs2_select_from_scores
  size_t off_part_o, off_part_ml, off_stats, off_scores, off_hist, off_state, off_bitmap, off_ckey, off_cidx, off_logits;
  size_t fa_bytes;
};

struct SaPlan {
  int RT, TG, split, nsplit, n_slots;
  size_t off_part_o, off_part_ml, bytes;
};

hs2_status check_dims(const hs2_dims* d) {
  if (!d) return fail(HS2_ERR_NULL, "dims is NULL");
  if (d->batch < 1 || d->n_q_heads < 1 || d->n_kv_heads < 1)
    return fail(HS2_ERR_SHAPE, "batch, n_q_heads and n_kv_heads must be >= 1");
  if (d->n_queries < 1 || d->n_queries > kMaxQueries)
    return fail(HS2_ERR_SHAPE, "n_queries must be in [1, %d] (got %d)", kMaxQueries, d->n_queries);
  if (d->n_q_heads % d->n_kv_heads)
    return fail(HS2_ERR_SHAPE, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)", d->n_q_heads, d->n_kv_heads);
  if (d->max_len < 1 || d->max_len > kMaxLen) return fail(HS2_ERR_SHAPE, "max_len must be in [1, 2^27]");
  if (d->head_dim != 128 && d->head_dim != 256)
    return fail(HS2_ERR_UNSUPPORTED, "head_dim %d not supported (128 or 256)", d->head_dim);
  const int G = d->n_q_heads / d->n_kv_heads;
  if (G > kMaxGroup) return fail(HS2_ERR_UNSUPPORTED, "query heads per KV head %d > %d", G, kMaxGroup);
  // one grid row per (b, g, c) in the selection and sparse kernels
  if ((int64_t)d->batch * d->n_kv_heads * d->n_queries > kMaxGridRows)
    return fail(HS2_ERR_UNSUPPORTED, "batch * n_kv_heads * n_queries exceeds %d", kMaxGridRows);
  if (d->n_queries * next_pow2(G) > kMaxRows)
    return fail(HS2_ERR_UNSUPPORTED, "n_queries * pow2(G) = %d exceeds %d query rows per KV head",
                d->n_queries * next_pow2(G), kMaxRows);
  if (d->kv_stride_t < d->head_dim || d->kv_stride_t % 8 || d->kv_stride_h < 0 || d->kv_stride_h % 8 ||
      d->kv_stride_b < 0 || d->kv_stride_b % 8)
    return fail(HS2_ERR_ALIGN, "KV strides must be non-negative multiples of 8 elements, kv_stride_t >= head_dim");
  // the streaming kernels address a tile of up to 64 token rows by 32-bit offsets
  if (d->kv_stride_t > kMaxTokenStride)
    return fail(HS2_ERR_UNSUPPORTED, "kv_stride_t %lld exceeds %lld elements", (long long)d->kv_stride_t,
                (long long)kMaxTokenStride);
  if (!std::isfinite(d->scale)) return fail(HS2_ERR_SHAPE, "scale must be finite");
  return HS2_OK;
}

hs2_status check_budget(int32_t k, int32_t window) {
  if (k < 0 || window < 0) return fail(HS2_ERR_SHAPE, "k and window must be >= 0");
  if ((int64_t)k + window < 1) return fail(HS2_ERR_SHAPE, "k + window must be >= 1");
  if ((int64_t)k + window > kMaxLen) return fail(HS2_ERR_SHAPE, "k + window too large");
  return HS2_OK;
}

size_t carve(size_t& cur, size_t bytes) {
  cur = (size_t)round_up((int64_t)cur, kAlign);
  const size_t at = cur;
  cur += bytes;
  return at;
}

// What the planner needs to know about the current device: compute units
// and, per full-attention kernel shape, how many workgroups stay resident
// on one compute unit (runtime occupancy query).
struct DeviceInfo {
  int cus = 256;
  int fa_wgs[2][4][kFaVariants] = {};  // [E4M3 cache][log2 RT][variant]; 0 = unknown
  int pool_wgs[2][2][4][7][17] = {};   // k_pool: [head dim 256][E4M3 cache][log2 RT][log2 Gp][C]; 0 = unknown
  void* scratch = nullptr;             // this device's address of `scratch` (hs2_sparse_attn_noalloc)
};

// Scratch of the allocation-free sparse layer (hs2_sparse_attn_noalloc): its
// split partials.  Every GPU the library runs on holds its own copy of this
// array, at its own address, until the process ends; host code never uses
// the array's name as a device address (it is a host-side stand-in), only
// the address hipGetSymbolAddress gives for the current device.
constexpr size_t kStaticScratchBytes = 16u << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

int ilog2(int v) {
  int l = 0;
  while ((1 << (l + 1)) <= v) ++l;
  return l;
}

// Measured on MI355X with one-round splits: 32-token tiles in 3 stages for
// one row tile; 16-token tiles in 3 stages and two token groups merged in
// LDS (half the split partials) for two; for four, one row tile per wave
// (four waves), 32-token tiles in 2 stages and two token groups; the
// workgroup kernel for eight.  Head dim 256: one row tile per wave, four
// row tiles in 32-token tiles and 2 stages, fewer in 16-token tiles and 3
// stages.  The one-row-tile shape serves both cache formats (E4M3 at 512K:
// 0.624 ms per step against 0.639 with 16-token tiles in 3 stages, whose
// stored logits also make the score pass slower, 69 against 59 us).
int default_fa_variant(int RT, int hd, bool kv8) {
  if (hd == 256) return RT >= 4 ? 8 : 6;
  if (RT >= 8) return kv8 ? 7 : 1;
  if (RT == 1) return 2;
  if (RT == 4) return 7;
  return 5;
}

// kv8: the cache is E4M3 (ring kernels only)
void make_plan(const hs2_dims* d, int32_t k, int32_t window, Plan& p, const DeviceInfo* di, bool kv8 = false) {
  p.kv8 = kv8;
  p.B = d->batch;
  p.C = d->n_queries;
  p.Hq = d->n_q_heads;
  p.Hkv = d->n_kv_heads;
  p.G = p.Hq / p.Hkv;
  p.Gp = next_pow2(p.G);
  p.D = d->head_dim;
  p.Lmax = d->max_len;
  p.k = k;
  p.W = window;
  p.S = k + window;
  const double scale = d->scale > 0.f ? (double)d->scale : 1.0 / std::sqrt((double)d->head_dim);
  p.c2 = (float)(scale * 1.4426950408889634);
  const int rows16 = (int)cdiv(p.C * p.Gp, 16);
  p.RT = next_pow2(rows16);
  p.fa_variant = env_int("HS2_FA_VARIANT", default_fa_variant(p.RT, p.D, kv8));
  if (p.fa_variant < 0 || p.fa_variant >= kFaVariants || fa_variant_head_dim(p.RT, p.fa_variant, kv8) != p.D)
    p.fa_variant = default_fa_variant(p.RT, p.D, kv8);
  p.TG = fa_token_groups(p.RT, p.fa_variant);
  p.units = (int64_t)p.B * p.Hkv;
  p.rows = p.units * p.C;
  // token splits: one item (sequence, KV head, split) per workgroup of a
  // grid of as many workgroups as stay resident at once on the device (one
  // round, no tail); the kernels derive the split length from the lengths
  // on the device (the shortest whose items fill the grid: ragged lengths
  // balance), a whole number of the kernel's token groups of 64-token tiles
  // and at least 256 tokens (a split's partial costs 16 RT rows of D + 4
  // floats).  HS2_FA_SPLIT fixes the length instead (grid: every split of
  // the capacity).
  const int lrt = p.RT >= 8 ? 3 : p.RT >= 4 ? 2 : p.RT >= 2 ? 1 : 0;
  const int wgs_cu = di && di->fa_wgs[kv8][lrt][p.fa_variant] > 0 ? di->fa_wgs[kv8][lrt][p.fa_variant] : 4;
  const int64_t slots = (int64_t)(di ? di->cus : 256) * wgs_cu * std::max(1, env_int("HS2_FA_ROUNDS", 1));
  const int align = fa_split_align(p.RT, p.fa_variant);
  p.fa_sp.align = align;
  p.fa_sp.min_split = (int)round_up(256, align);
  const int fixed = env_int("HS2_FA_SPLIT", 0);
  if (fixed > 0) {
    p.fa_sp.fixed = (int)std::max<int64_t>(align, round_up(std::min<int64_t>(fixed, p.Lmax), align));
    p.fa_sp.n_items = (int)(p.units * cdiv(p.Lmax, p.fa_sp.fixed));
  } else {
    p.fa_sp.fixed = 0;
    p.fa_sp.n_items = (int)std::max<int64_t>(slots, p.units);
  }
  // score pass over K: the same one-round rule for its own kernel; at most
  // 32768 tokens per split (16-bit histogram counters in LDS)
  const int pool_cu = di && p.C <= 16 ? di->pool_wgs[p.D == 256][kv8][lrt][ilog2(p.Gp)][p.C] : 0;
  const int64_t pslots = (int64_t)(di ? di->cus : 256) * (pool_cu > 0 ? pool_cu : 4);
  int psplit = (int)std::max<int64_t>(256, round_up(cdiv(p.Lmax, std::max<int64_t>(1, pslots / p.units)), 64));
  psplit = env_int("HS2_POOL_SPLIT", psplit);
  psplit = (int)std::max<int64_t>(64, round_up(std::min<int64_t>(std::min(psplit, 32768), p.Lmax), 64));
  p.pool_split = psplit;
  p.pool_nsplit = (int)cdiv(p.Lmax, psplit);
  p.score_stride = round_up(p.Lmax, 64);
  p.bitmap_words = cdiv(p.Lmax, 64);
  p.cand_cap = p.Lmax;
  p.sel_nchunks = (int)cdiv(p.Lmax, kSelChunk);
  // with at most 16 query rows per KV head (C * G <= 16) the ring kernel
  // stores its logits (4 C G bytes per token) and the scores are computed
  // from them instead of re-reading K (256 bytes per token)
  p.pool_logits = p.RT == 1 && p.fa_variant != 1 && env_int("HS2_POOL_FROM_K", 0) == 0;
  p.logit_stride = round_up(p.Lmax, 64);
  // Cache policy of the full-attention ring kernel's loads.  A cache that
  // fits the last-level cache keeps every row cacheable (a decode loop finds
  // it there again).  A larger one streams V.  K streams too where the scores
  // come from the stored logits; where the score pass re-reads K, the last
  // kFaKeepPercent (HS2_FA_K_KEEP) percent of each token group's K rows stay
  // cacheable for it (it walks each split from the end); one row tile keeps
  // all of K then (no per-tile policy switch).
  {
    const int64_t kv_bytes = 2 * (int64_t)p.B * p.Hkv * p.Lmax * p.D * (kv8 ? 1 : 2);
    const bool stream = kv_bytes > kLastLevelCacheBytes;
    // the kernel keeps the last `keep` percent of each token group's part of
    // its split cacheable (a ring kernel with two token groups streams two
    // such parts per split) and streams the K rows before them
    int keep = kFaKeepPercent;
    const int ek = env_int("HS2_FA_K_KEEP", -1);
    if (ek >= 0 && ek <= 100) keep = ek;
    p.fa_cache_policy = !stream ? FA_CACHE_DEFAULT
                        : p.RT == 1 ? (p.pool_logits ? FA_STREAM_KV : FA_STREAM_V)
                                    : FA_STREAM_K_HEAD;
    p.fa_k_keep = keep;
    const int ep = env_int("HS2_FA_CACHE_POLICY", -1);
    if (ep >= 0 && fa_cache_policy_built(p.RT, ep)) p.fa_cache_policy = ep;
  }
  // score pass over stored logits: chunks of 1024-4096 tokens (whole float4
  // steps of its 256 threads), about two workgroups per CU
  p.logit_chunk = (int)std::min<int64_t>(
      4096, std::max<int64_t>(1024, round_up(cdiv(p.Lmax * p.units, 2 * (int64_t)(di ? di->cus : 256)), 1024)));

  const int64_t prow = 16 * p.RT;
  const int64_t nslot = (int64_t)p.fa_sp.n_items * p.TG;  // partial slots of the full-attention pass
  size_t cur = 0;
  p.off_part_o = carve(cur, sizeof(float) * nslot * prow * p.D);
  p.off_part_ml = carve(cur, sizeof(float) * nslot * prow * 4);
  p.off_stats = carve(cur, sizeof(float) * (size_t)p.B * p.C * p.Hq * 2);
  p.off_scores = carve(cur, sizeof(float) * p.rows * p.score_stride);
  p.off_hist = carve(cur, sizeof(uint32_t) * p.rows * kNBins);
  p.off_state = carve(cur, sizeof(int32_t) * p.rows * 8);
  p.off_bitmap = carve(cur, sizeof(uint64_t) * p.rows * p.bitmap_words);
  p.off_ckey = carve(cur, sizeof(uint32_t) * p.rows * p.cand_cap);
  p.off_cidx = carve(cur, sizeof(int32_t) * p.rows * p.cand_cap);
  p.off_logits = carve(cur, p.pool_logits ? sizeof(float) * p.rows * p.G * p.logit_stride : 0);
  p.fa_bytes = (size_t)round_up((int64_t)cur, kAlign);
}

void make_sa_plan(const Plan& p, int n_slots, SaPlan& s) {
  s.n_slots = n_slots;
  s.RT = next_pow2((int)cdiv(p.Gp, 16));
  s.TG = 1;  // one partial per split
  // about 1024 workgroups, at most 4096 slots each (their indices are staged in LDS)
  int split = (int)std::max<int64_t>(64, round_up(cdiv(p.rows * (int64_t)n_slots, 1024), 64));
  split = env_int("HS2_SA_SPLIT", split);
  split = (int)std::min<int64_t>(4096, std::max<int64_t>(64, round_up(std::min<int64_t>(split, n_slots), 64)));
  s.split = split;
  s.nsplit = (int)cdiv(n_slots, split);
  const int64_t prow = 16 * s.RT;
  size_t cur = 0;
  s.off_part_o = carve(cur, sizeof(float) * p.rows * s.nsplit * s.TG * prow * p.D);
  s.off_part_ml = carve(cur, sizeof(float) * p.rows * s.nsplit * s.TG * prow * 4);
  s.bytes = (size_t)round_up((int64_t)cur, kAlign);
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// ---------------------------------------------------------------- timing
enum KernelKind { KK_FA = 0, KK_COMBINE, KK_POOL, KK_POOL_LOGITS, KK_SEL_INIT, KK_SEL_HIST, KK_SELECT,
                  KK_BLOCK_SELECT, KK_SA, KK_SA_COMBINE, KK_COUNT };
const char* kKindNames[KK_COUNT] = {"fa_split", "fa_combine", "pool_scores", "pool_logits", "sel_init", "sel_hist",
                                    "select", "block_select", "sa_split", "sa_combine"};
constexpr int kMaxTimed = 16384;
struct Timing {
  bool on = false;
  int n = 0;
  std::vector<hipEvent_t> ev0, ev1;
  std::vector<int> kind;
} g_timing;

struct TimedLaunch {
  hipStream_t s;
  int slot = -1;
  TimedLaunch(KernelKind kk, hipStream_t st) : s(st) {
    if (g_timing.on && g_timing.n < (int)g_timing.ev0.size()) {
      slot = g_timing.n++;
      g_timing.kind[slot] = kk;
      (void)hipEventRecord(g_timing.ev0[slot], s);
    }
  }
  ~TimedLaunch() {
    if (slot >= 0) (void)hipEventRecord(g_timing.ev1[slot], s);
  }
};

std::mutex g_init_mu;
bool g_dev_done[64] = {};
DeviceInfo g_dev[64];

// Per-device set-up (once, with that device current): LDS limits of the
// kernels that need more than 64 KB, the occupancy figures the planner
// uses, and this device's address of the static scratch array.
hs2_status ensure_device_init(const DeviceInfo** info) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(HS2_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= 64) return fail(HS2_ERR_HIP, "device index out of range");
  std::lock_guard<std::mutex> lk(g_init_mu);
  if (!g_dev_done[dev]) {
    hipError_t e = set_pool_smem_limits();
    if (e != hipSuccess) return fail(HS2_ERR_HIP, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    DeviceInfo di;
    if ((e = hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
      return fail(HS2_ERR_HIP, "hipDeviceGetAttribute: %s", hipGetErrorString(e));
    for (int f = 0; f < 2; ++f)
      for (int l = 0; l < 4; ++l) {
        for (int v = 0; v < kFaVariants; ++v)
          if ((e = fa_wgs_per_cu(1 << l, v, f == 1, &di.fa_wgs[f][l][v])) != hipSuccess)
            return fail(HS2_ERR_HIP, "occupancy query: %s", hipGetErrorString(e));
        for (int h = 0; h < 2; ++h)
          for (int lg = 0; lg < 7; ++lg)
            for (int c = 1; c <= 16; ++c)
              if ((e = pool_wgs_per_cu(1 << l, 1 << lg, c, f == 1, h ? 256 : 128, &di.pool_wgs[h][f][l][lg][c])) !=
                  hipSuccess)
                return fail(HS2_ERR_HIP, "occupancy query: %s", hipGetErrorString(e));
      }
    if ((e = hipGetSymbolAddress(&di.scratch, HIP_SYMBOL(scratch))) != hipSuccess || !di.scratch)
      return fail(HS2_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_dev[dev] = di;
    g_dev_done[dev] = true;
  }
  if (info) *info = &g_dev[dev];
  return HS2_OK;
}

// Device information for planning if a device is present (null on a host
// without one; the plan then falls back to fixed figures).
const DeviceInfo* try_device_info() {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) return nullptr;
  const DeviceInfo* di = nullptr;
  return ensure_device_init(&di) == HS2_OK ? di : nullptr;
}

#define HS2_TRY_LAUNCH(kind, stream, call)                                                        \
  do {                                                                                              \
    hipError_t e_;                                                                                  \
    {                                                                                               \
      TimedLaunch tl_(kind, stream);                                                                \
      e_ = (call);                                                                                  \
    }                                                                                               \
    if (e_ != hipSuccess) return fail(HS2_ERR_HIP, "%s launch: %s", kKindNames[kind], hipGetErrorString(e_)); \
  } while (0)

SelArgs sel_args(const Plan& p, char* ws, const float* scores, int64_t score_stride, const int32_t* len,
                 int32_t* idx) {
  SelArgs a{};
  a.scores = scores;
  a.len = len;
  a.hist = (uint32_t*)(ws + p.off_hist);
  a.state = (int32_t*)(ws + p.off_state);
  a.bitmap = (uint64_t*)(ws + p.off_bitmap);
  a.cand_key = (uint32_t*)(ws + p.off_ckey);
  a.cand_idx = (int32_t*)(ws + p.off_cidx);
  a.idx = idx;
  a.rows = p.rows;
  a.score_stride = score_stride;
  a.bitmap_words = p.bitmap_words;
  a.cand_cap = p.cand_cap;
  a.B = p.B;
  a.C = p.C;
  a.Hkv = p.Hkv;
  a.max_len = p.Lmax;
  a.k = p.k;
  a.W = p.W;
  a.S = p.S;
  a.chunk = kSelChunk;
  return a;
}

hs2_status run_selection_tail(const Plan& p, const SelArgs& sa, hipStream_t s) {
  HS2_TRY_LAUNCH(KK_SELECT, s, launch_select(sa, s));
  return HS2_OK;
}

}  // namespace

extern "C" {

const char* hs2_status_string(int32_t status) {
  switch (status) {
    case HS2_OK: return "ok";
    case HS2_ERR_NULL: return "required pointer is NULL";
    case HS2_ERR_SHAPE: return "invalid dimensions or budgets";
    case HS2_ERR_UNSUPPORTED: return "unsupported configuration";
    case HS2_ERR_WORKSPACE: return "workspace too small";
    case HS2_ERR_ALIGN: return "pointer or stride misaligned";
    case HS2_ERR_HIP: return "HIP runtime or launch failure";
    default: return "unknown status";
  }
}

const char* hs2_last_error(void) { return g_last_error.c_str(); }

size_t hs2_workspace_bytes(const hs2_dims* dims, int32_t k, int32_t window) {
  if (check_dims(dims) != HS2_OK || check_budget(k, window) != HS2_OK) return 0;
  const DeviceInfo* di = try_device_info();
  size_t bytes = 0;
  for (int kv8 = 0; kv8 < 2; ++kv8) {  // enough for either cache format
    Plan p;
    make_plan(dims, k, window, p, di, kv8 == 1);
    SaPlan sp;
    make_sa_plan(p, k + window, sp);
    bytes = std::max(bytes, std::max(p.fa_bytes, sp.bytes));
  }
  return bytes;
}

}  // extern "C"

namespace {

// E4M3 cache: K and V are byte arrays with one float scale per KV head each;
// their strides must keep every 16-byte load aligned
hs2_status check_fp8(const hs2_dims* dims, const float* k_scale, const float* v_scale) {
  if (!k_scale || !v_scale) return fail(HS2_ERR_NULL, "k_scale and v_scale are required for an FP8 cache");
  if (!aligned(k_scale, 4) || !aligned(v_scale, 4)) return fail(HS2_ERR_ALIGN, "scales need 4-byte alignment");
  if (dims->kv_stride_t % 16 || dims->kv_stride_h % 16 || dims->kv_stride_b % 16)
    return fail(HS2_ERR_ALIGN, "FP8 cache strides must be multiples of 16 elements");
  return HS2_OK;
}

// block-level selection: blocks of a power-of-two size in [16, 256], k a
// whole number of blocks, at most 16384 blocks per row (their keys sit in LDS)
hs2_status check_block(const hs2_dims* d, int32_t k, int32_t block) {
  if (block < 16 || block > 256 || (block & (block - 1)))
    return fail(HS2_ERR_SHAPE, "block must be a power of two in [16, 256] (got %d)", block);
  if (k % block) return fail(HS2_ERR_SHAPE, "k (%d) must be a multiple of block (%d)", k, block);
  if (((int64_t)d->max_len + block - 1) / block > 16384)
    return fail(HS2_ERR_UNSUPPORTED, "max_len / block exceeds 16384 blocks");
  return HS2_OK;
}

// block keys go to the token candidates' region of the workspace (unused by
// block-level selection; rows x max_len keys >= rows x blocks)
BlockSelArgs block_sel_args(const Plan& p, char* ws, const float* scores, int64_t score_stride, const int32_t* len,
                            int32_t* idx, int block) {
  BlockSelArgs a{};
  a.scores = scores;
  a.len = len;
  a.idx = idx;
  a.keys = (uint32_t*)(ws + p.off_ckey);
  a.key_stride = ((int64_t)p.Lmax + block - 1) / block;
  a.rows = p.rows;
  a.score_stride = score_stride;
  a.C = p.C;
  a.Hkv = p.Hkv;
  a.max_len = p.Lmax;
  a.k = p.k;
  a.W = p.W;
  a.S = p.S;
  a.block = block;
  return a;
}

// block == 0: token-level selection
hs2_status full_attn_impl(const hs2_dims* dims, const uint16_t* q, const void* K, const void* V, const float* k_scale,
                          const float* v_scale, const int32_t* len, int32_t k, int32_t window, int32_t block,
                          uint16_t* out, int32_t* idx, float* stats, float* scores, void* workspace,
                          size_t workspace_bytes, void* stream) {
  const bool kv8 = k_scale != nullptr;
  hs2_status st = check_dims(dims);
  if (st != HS2_OK) return st;
  if ((st = check_budget(k, window)) != HS2_OK) return st;
  if (kv8 && (st = check_fp8(dims, k_scale, v_scale)) != HS2_OK) return st;
  if (block && (st = check_block(dims, k, block)) != HS2_OK) return st;
  if (!q || !K || !V || !len || !out || !idx || !workspace)
    return fail(HS2_ERR_NULL, "q, K, V, len, out, idx and workspace are required");
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16) || !aligned(idx, 4) ||
      !aligned(len, 4) || !aligned(workspace, kAlign) || (stats && !aligned(stats, 8)) || (scores && !aligned(scores, 4)))
    return fail(HS2_ERR_ALIGN, "q/K/V/out need 16-byte, workspace 256-byte, idx/len/scores 4-byte alignment");
  const DeviceInfo* di = try_device_info();
  Plan p;
  make_plan(dims, k, window, p, di, kv8);
  if (workspace_bytes < p.fa_bytes)
    return fail(HS2_ERR_WORKSPACE, "workspace %zu bytes < %zu required", workspace_bytes, p.fa_bytes);
  if ((st = ensure_device_init(&di)) != HS2_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  float* stats_log2 = (float*)(ws + p.off_stats);
  float* sc = scores ? scores : (float*)(ws + p.off_scores);
  const int64_t sc_stride = scores ? (int64_t)p.Lmax : p.score_stride;

  SelArgs sa = sel_args(p, ws, sc, sc_stride, len, idx);

  FaArgs fa{};
  fa.q = q;
  fa.K = (const uint16_t*)K;
  fa.V = (const uint16_t*)V;
  fa.k_scale = k_scale;
  fa.len = len;
  fa.part_o = (float*)(ws + p.off_part_o);
  fa.part_ml = (float*)(ws + p.off_part_ml);
  fa.stride_b = dims->kv_stride_b;
  fa.stride_h = dims->kv_stride_h;
  fa.stride_t = dims->kv_stride_t;
  fa.c2 = p.c2;
  fa.B = p.B;
  fa.C = p.C;
  fa.Hq = p.Hq;
  fa.Hkv = p.Hkv;
  fa.G = p.G;
  fa.Gp = p.Gp;
  fa.max_len = p.Lmax;
  fa.sp = p.fa_sp;
  fa.logits = p.pool_logits ? (float*)(ws + p.off_logits) : nullptr;
  fa.logit_stride = p.logit_stride;
  fa.cache_policy = p.fa_cache_policy;
  fa.k_keep_pct = p.fa_k_keep;
  HS2_TRY_LAUNCH(KK_FA, s, launch_fa_split(fa, p.RT, p.fa_variant, s));

  CombineArgs ca{};
  ca.part_o = fa.part_o;
  ca.part_ml = fa.part_ml;
  ca.len = len;
  ca.out = out;
  ca.stats_log2 = stats_log2;
  ca.stats_user = stats;
  ca.B = p.B;
  ca.C = p.C;
  ca.Hq = p.Hq;
  ca.Hkv = p.Hkv;
  ca.G = p.G;
  ca.Gp = p.Gp;
  ca.max_len = p.Lmax;
  ca.rows = 16 * p.RT;
  ca.nslot = 0;  // per (sequence, KV head): derived in the kernel from the splits
  ca.tg = p.TG;
  ca.sp = p.fa_sp;
  ca.sa_mode = 0;
  // the histogram and the per-row counters (contiguous) start at zero
  ca.v_scale = v_scale;
  ca.hd = p.D;
  ca.clear = block ? nullptr : (uint4*)(ws + p.off_hist);
  ca.n_clear = (int64_t)(p.off_state - p.off_hist + sizeof(int32_t) * p.rows * 8) / 16;
  HS2_TRY_LAUNCH(KK_COMBINE, s, launch_combine(ca, std::min(16 * p.RT, p.C * p.Gp), p.units, s));

  PoolArgs pa{};
  pa.q = q;
  pa.K = (const uint16_t*)K;
  pa.k_scale = k_scale;
  pa.hd = p.D;
  pa.len = len;
  pa.stats_log2 = stats_log2;
  pa.scores = sc;
  pa.hist = block ? nullptr : sa.hist;  // block selection needs no histogram
  pa.stride_b = dims->kv_stride_b;
  pa.stride_h = dims->kv_stride_h;
  pa.stride_t = dims->kv_stride_t;
  pa.score_stride = sc_stride;
  pa.c2 = p.c2;
  pa.B = p.B;
  pa.C = p.C;
  pa.Hq = p.Hq;
  pa.Hkv = p.Hkv;
  pa.G = p.G;
  pa.Gp = p.Gp;
  pa.max_len = p.Lmax;
  pa.W = p.W;
  pa.split_tokens = p.pool_logits ? p.logit_chunk : p.pool_split;
  pa.n_split = p.pool_nsplit;
  pa.logits = fa.logits;
  pa.logit_stride = p.logit_stride;
  pa.k_stream = p.fa_cache_policy != FA_CACHE_DEFAULT;
  if (p.pool_logits)
    HS2_TRY_LAUNCH(KK_POOL_LOGITS, s, launch_pool_logits(pa, s));
  else
    HS2_TRY_LAUNCH(KK_POOL, s, launch_pool(pa, p.RT, s));
  if (block) {
    const BlockSelArgs ba = block_sel_args(p, ws, sc, sc_stride, len, idx, block);
    HS2_TRY_LAUNCH(KK_BLOCK_SELECT, s, launch_block_select(ba, s));
    return HS2_OK;
  }
  return run_selection_tail(p, sa, s);
}

}  // namespace

extern "C" {

hs2_status hs2_full_attn_score_select(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                      const int32_t* len, int32_t k, int32_t window, uint16_t* out, int32_t* idx,
                                      float* stats, float* scores, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  return full_attn_impl(dims, q, K, V, nullptr, nullptr, len, k, window, 0, out, idx, stats, scores, workspace,
                        workspace_bytes, stream);
}

hs2_status hs2_full_attn_score_select_blocks(const hs2_dims* dims, const uint16_t* q, const uint16_t* K,
                                             const uint16_t* V, const int32_t* len, int32_t k, int32_t window,
                                             int32_t block, uint16_t* out, int32_t* idx, float* stats,
                                             float* scores, void* workspace, size_t workspace_bytes,
                                             void* stream) {
  if (block == 0) return fail(HS2_ERR_SHAPE, "block must be a power of two in [16, 256] (got 0)");
  return full_attn_impl(dims, q, K, V, nullptr, nullptr, len, k, window, block, out, idx, stats, scores, workspace,
                        workspace_bytes, stream);
}

hs2_status hs2_full_attn_score_select_fp8(const hs2_dims* dims, const uint16_t* q, const uint8_t* K,
                                          const uint8_t* V, const float* k_scale, const float* v_scale,
                                          const int32_t* len, int32_t k, int32_t window, uint16_t* out,
                                          int32_t* idx, float* stats, float* scores, void* workspace,
                                          size_t workspace_bytes, void* stream) {
  if (!k_scale || !v_scale) return fail(HS2_ERR_NULL, "k_scale and v_scale are required for an FP8 cache");
  return full_attn_impl(dims, q, K, V, k_scale, v_scale, len, k, window, 0, out, idx, stats, scores, workspace,
                        workspace_bytes, stream);
}

hs2_status hs2_select_from_scores(const hs2_dims* dims, const float* scores, const int32_t* len, int32_t k,
                                  int32_t window, int32_t* idx, void* workspace, size_t workspace_bytes, void* stream) {
  hs2_status st = check_dims(dims);
  if (st != HS2_OK) return st;
  if ((st = check_budget(k, window)) != HS2_OK) return st;
  if (!scores || !len || !idx || !workspace) return fail(HS2_ERR_NULL, "scores, len, idx and workspace are required");
  if (!aligned(scores, 4) || !aligned(len, 4) || !aligned(idx, 4) || !aligned(workspace, kAlign))
    return fail(HS2_ERR_ALIGN, "scores/len/idx need 4-byte, workspace 256-byte alignment");
  const DeviceInfo* di = try_device_info();
  Plan p;
  make_plan(dims, k, window, p, di);
  if (workspace_bytes < p.fa_bytes)
    return fail(HS2_ERR_WORKSPACE, "workspace %zu bytes < %zu required", workspace_bytes, p.fa_bytes);
  if ((st = ensure_device_init(&di)) != HS2_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  SelArgs sa = sel_args(p, (char*)workspace, scores, p.Lmax, len, idx);
  HS2_TRY_LAUNCH(KK_SEL_INIT, s, launch_sel_init(sa, s));
  HS2_TRY_LAUNCH(KK_SEL_HIST, s, launch_sel_hist(sa, p.sel_nchunks, s));
  return run_selection_tail(p, sa, s);
}

hs2_status hs2_select_blocks_from_scores(const hs2_dims* dims, const float* scores, const int32_t* len, int32_t k,
                                         int32_t window, int32_t block, int32_t* idx, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  hs2_status st = check_dims(dims);
  if (st != HS2_OK) return st;
  if ((st = check_budget(k, window)) != HS2_OK) return st;
  if ((st = check_block(dims, k, block)) != HS2_OK) return st;
  if (!scores || !len || !idx || !workspace) return fail(HS2_ERR_NULL, "scores, len, idx and workspace are required");
  if (!aligned(scores, 4) || !aligned(len, 4) || !aligned(idx, 4) || !aligned(workspace, kAlign))
    return fail(HS2_ERR_ALIGN, "scores/len/idx need 4-byte, workspace 256-byte alignment");
  const DeviceInfo* di = try_device_info();
  Plan p;
  make_plan(dims, k, window, p, di);
  if (workspace_bytes < p.fa_bytes)
    return fail(HS2_ERR_WORKSPACE, "workspace %zu bytes < %zu required", workspace_bytes, p.fa_bytes);
  if ((st = ensure_device_init(&di)) != HS2_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const BlockSelArgs ba = block_sel_args(p, (char*)workspace, scores, p.Lmax, len, idx, block);
  HS2_TRY_LAUNCH(KK_BLOCK_SELECT, s, launch_block_select(ba, s));
  return HS2_OK;
}

hs2_status hs2_sparse_attn(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                           const int32_t* len, const int32_t* idx, int32_t n_slots, uint16_t* out, void* workspace,
                           size_t workspace_bytes, void* stream) {
  return hs2_sparse_attn_ex(dims, q, K, V, len, idx, n_slots, nullptr, nullptr, out, workspace, workspace_bytes,
                            stream);
}

}  // extern "C"

namespace {

hs2_status sparse_impl(const hs2_dims* dims, const uint16_t* q, const void* K, const void* V, const float* k_scale,
                       const float* v_scale, const int32_t* len, const int32_t* idx, int32_t n_slots,
                       const float* sink, const uint16_t* gate, uint16_t* out, void* workspace,
                       size_t workspace_bytes, void* stream) {
  const bool kv8 = k_scale != nullptr;
  hs2_status st = check_dims(dims);
  if (st != HS2_OK) return st;
  if (n_slots < 1 || n_slots > kMaxLen) return fail(HS2_ERR_SHAPE, "n_slots must be in [1, 2^27]");
  if (kv8 && (st = check_fp8(dims, k_scale, v_scale)) != HS2_OK) return st;
  if (!q || !K || !V || !len || !idx || !out || !workspace)
    return fail(HS2_ERR_NULL, "q, K, V, len, idx, out and workspace are required");
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(out, 16) || !aligned(idx, 4) ||
      !aligned(len, 4) || !aligned(workspace, kAlign) || (sink && !aligned(sink, 4)) || (gate && !aligned(gate, 8)))
    return fail(HS2_ERR_ALIGN,
                "q/K/V/out need 16-byte, workspace 256-byte, gate 8-byte, idx/len/sink 4-byte alignment");
  const DeviceInfo* di = try_device_info();
  Plan p;
  make_plan(dims, 0, n_slots, p, di, kv8);
  SaPlan sp;
  make_sa_plan(p, n_slots, sp);
  if (workspace_bytes < sp.bytes)
    return fail(HS2_ERR_WORKSPACE, "workspace %zu bytes < %zu required", workspace_bytes, sp.bytes);
  if ((st = ensure_device_init(&di)) != HS2_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  SaArgs a{};
  a.q = q;
  a.K = (const uint16_t*)K;
  a.V = (const uint16_t*)V;
  a.k_scale = k_scale;
  a.hd = p.D;
  a.len = len;
  a.idx = idx;
  a.part_o = (float*)(ws + sp.off_part_o);
  a.part_ml = (float*)(ws + sp.off_part_ml);
  a.stride_b = dims->kv_stride_b;
  a.stride_h = dims->kv_stride_h;
  a.stride_t = dims->kv_stride_t;
  a.idx_stride = n_slots;
  a.c2 = p.c2;
  a.B = p.B;
  a.C = p.C;
  a.Hq = p.Hq;
  a.Hkv = p.Hkv;
  a.G = p.G;
  a.max_len = p.Lmax;
  a.n_slots = n_slots;
  a.split_slots = sp.split;
  a.n_split = sp.nsplit;
  HS2_TRY_LAUNCH(KK_SA, s, launch_sa_split(a, sp.RT, s));

  CombineArgs ca{};
  ca.part_o = a.part_o;
  ca.part_ml = a.part_ml;
  ca.len = len;
  ca.out = out;
  ca.stats_log2 = nullptr;
  ca.stats_user = nullptr;
  ca.B = p.B;
  ca.C = p.C;
  ca.Hq = p.Hq;
  ca.Hkv = p.Hkv;
  ca.G = p.G;
  ca.Gp = p.Gp;
  ca.max_len = p.Lmax;
  ca.rows = 16 * sp.RT;
  ca.nslot = sp.nsplit * sp.TG;
  ca.tg = sp.TG;
  ca.sa_mode = 1;
  ca.sink = sink;
  ca.gate = gate;
  ca.v_scale = v_scale;
  ca.hd = p.D;
  HS2_TRY_LAUNCH(KK_SA_COMBINE, s, launch_combine(ca, p.G, p.rows, s));
  return HS2_OK;
}

}  // namespace

extern "C" {

hs2_status hs2_sparse_attn_ex(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                              const int32_t* len, const int32_t* idx, int32_t n_slots, const float* sink,
                              const uint16_t* gate, uint16_t* out, void* workspace, size_t workspace_bytes,
                              void* stream) {
  return sparse_impl(dims, q, K, V, nullptr, nullptr, len, idx, n_slots, sink, gate, out, workspace,
                     workspace_bytes, stream);
}

hs2_status hs2_sparse_attn_noalloc(const hs2_dims* dims, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                                   const int32_t* len, const int32_t* idx, int32_t n_slots, uint16_t* out,
                                   void* stream) {
  hs2_status st = check_dims(dims);
  if (st != HS2_OK) return st;
  if (n_slots < 1 || n_slots > kMaxLen) return fail(HS2_ERR_SHAPE, "n_slots must be in [1, 2^27]");
  // the scratch this call needs, checked against the static array before
  // anything touches the device (the sparse plan needs no device figures)
  Plan p;
  make_plan(dims, 0, n_slots, p, nullptr, false);
  SaPlan sp;
  make_sa_plan(p, n_slots, sp);
  if (sp.bytes > kStaticScratchBytes)
    return fail(HS2_ERR_WORKSPACE, "sparse layer needs %zu bytes of scratch; the static scratch holds %zu",
                sp.bytes, kStaticScratchBytes);
  const DeviceInfo* di = nullptr;
  if ((st = ensure_device_init(&di)) != HS2_OK) return st;
  return sparse_impl(dims, q, K, V, nullptr, nullptr, len, idx, n_slots, nullptr, nullptr, out, di->scratch,
                     kStaticScratchBytes, stream);
}

hs2_status hs2_sparse_attn_fp8(const hs2_dims* dims, const uint16_t* q, const uint8_t* K, const uint8_t* V,
                               const float* k_scale, const float* v_scale, const int32_t* len, const int32_t* idx,
                               int32_t n_slots, const float* sink, const uint16_t* gate, uint16_t* out,
                               void* workspace, size_t workspace_bytes, void* stream) {
  if (!k_scale || !v_scale) return fail(HS2_ERR_NULL, "k_scale and v_scale are required for an FP8 cache");
  return sparse_impl(dims, q, K, V, k_scale, v_scale, len, idx, n_slots, sink, gate, out, workspace,
                     workspace_bytes, stream);
}

hs2_status hs2_stream_read_probe(const void* src, size_t bytes, int32_t mode, uint32_t* sink, void* stream) {
  if (!src || !sink) return fail(HS2_ERR_NULL, "src and sink are required");
  if (mode < 0 || mode > 5) return fail(HS2_ERR_SHAPE, "mode must be in [0, 5] (got %d)", mode);
  if (bytes == 0) return fail(HS2_ERR_SHAPE, "bytes must be > 0");
  const size_t rec = mode == 4 ? 512 : 256;  // gather modes: record bytes
  if (mode >= 4 && (bytes % rec || ((bytes / rec) & (bytes / rec - 1))))
    return fail(HS2_ERR_SHAPE, "mode %d reads %zu-byte records: bytes must be %zu times a power of two", mode, rec,
                rec);
  if (!aligned(src, 16) || bytes % 16 || !aligned(sink, 4))
    return fail(HS2_ERR_ALIGN, "src needs 16-byte alignment and a multiple of 16 bytes, sink 4-byte alignment");
  static_assert(HS2_STREAM_PROBE_SINK_WORDS == STREAM_PROBE_WORKGROUPS, "one sink word per probe workgroup");
  hipStream_t s = (hipStream_t)stream;
  const hipError_t e = launch_stream_probe(src, (int64_t)(bytes / 16), mode, sink, s);
  if (e != hipSuccess) return fail(HS2_ERR_HIP, "stream probe launch: %s", hipGetErrorString(e));
  return HS2_OK;
}

hs2_status hs2_timing_enable(int32_t on) {
  if (on && g_timing.ev0.empty()) {
    g_timing.ev0.resize(kMaxTimed);
    g_timing.ev1.resize(kMaxTimed);
    g_timing.kind.resize(kMaxTimed);
    for (int i = 0; i < kMaxTimed; ++i) {
      if (hipEventCreate(&g_timing.ev0[i]) != hipSuccess || hipEventCreate(&g_timing.ev1[i]) != hipSuccess) {
        g_timing.ev0.clear();
        g_timing.ev1.clear();
        g_timing.kind.clear();
        return fail(HS2_ERR_HIP, "hipEventCreate failed");
      }
    }
  }
  g_timing.on = on != 0;
  return HS2_OK;
}

void hs2_timing_reset(void) { g_timing.n = 0; }

int32_t hs2_timing_read(char* names, size_t names_len, int32_t* counts, double* total_ms, int32_t max_kernels) {
  double tot[KK_COUNT] = {};
  int cnt[KK_COUNT] = {};
  for (int i = 0; i < g_timing.n; ++i) {
    if (hipEventSynchronize(g_timing.ev1[i]) != hipSuccess) return fail(HS2_ERR_HIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g_timing.ev0[i], g_timing.ev1[i]) != hipSuccess)
      return fail(HS2_ERR_HIP, "hipEventElapsedTime failed");
    tot[g_timing.kind[i]] += ms;
    cnt[g_timing.kind[i]] += 1;
  }
  int n = 0;
  size_t pos = 0;
  for (int kk = 0; kk < KK_COUNT && n < max_kernels; ++kk) {
    if (!cnt[kk]) continue;
    const size_t L = strlen(kKindNames[kk]) + 1;
    if (names && pos + L <= names_len) {
      memcpy(names + pos, kKindNames[kk], L);
      pos += L;
    }
    if (counts) counts[n] = cnt[kk];
    if (total_ms) total_ms[n] = tot[kk];
    ++n;
  }
  return n;
}

}  // extern "C"
