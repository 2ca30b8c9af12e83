// Internal interface between the C ABI (hs2_api.hip) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hs2 {

// Token splits of the full-attention pass: fixed > 0 fixes the split
// length; else every workgroup derives the balanced length from len[] (the
// shortest multiple of align, at least min_split, whose (sequence, KV head,
// split) items number at most n_items, the grid size).
struct FaSplitPlan {
  int fixed, align, min_split, n_items;
};

struct FaArgs {
  const uint16_t* q;
  const uint16_t* K;
  const uint16_t* V;
  const int32_t* len;
  float* part_o;   // [n_items * TG][16 RT][HD]
  float* part_ml;  // [n_items * TG][16 RT][4]: (m ref, l, m true, 0)
  int64_t stride_b, stride_h, stride_t;
  float c2;        // softmax scale * log2(e)
  int B, C, Hq, Hkv, G, Gp, max_len;
  FaSplitPlan sp;  // grid: sp.n_items workgroups, one (sequence, KV head, split) item each
  float* logits;   // [B*Hkv][C*G][logit_stride] logits in log2 units (ring kernels), or null
  int64_t logit_stride;
  const float* k_scale;  // [Hkv] for an E4M3 cache (K, V are then byte arrays), else null
  int cache_policy;      // ring kernels: FaCachePolicy of the stage loads
  int k_keep_pct;        // FA_STREAM_K_HEAD: the last k_keep_pct % of each token group's K rows stay
                         // cacheable, the rows before them are non-temporal
};

// Cache policy of the full-attention ring kernel's loads.  Non-temporal
// rows stream past the caches: for rows read once, so that they do not
// evict lines a later pass reads again.
enum FaCachePolicy {
  FA_CACHE_DEFAULT = 0,  // every row cacheable
  FA_STREAM_V = 1,       // V non-temporal, K cacheable
  FA_STREAM_KV = 2,      // K and V non-temporal
  FA_STREAM_K_HEAD = 3,  // V non-temporal, K non-temporal in the leading part of each token group
};
// Policies built for each query row tile count: one row tile takes no
// per-tile branch (it is latency-sensitive), more row tiles take the split one.
constexpr bool fa_cache_policy_built(int rt, int kp) {
  return kp == FA_CACHE_DEFAULT || (rt == 1 ? (kp == FA_STREAM_V || kp == FA_STREAM_KV) : kp == FA_STREAM_K_HEAD);
}

struct CombineArgs {
  const float* part_o;
  const float* part_ml;
  const int32_t* len;
  uint16_t* out;        // [B, C, Hq, HD] bf16
  float* stats_log2;    // [B, C, Hq, 2] (reference max M in log2 units, Z against it) or null
  float* stats_user;    // [B, C, Hq, 2] (M in natural units, Z) or null
  int B, C, Hq, Hkv, G, Gp, max_len;
  int rows;             // partial rows per slot
  int nslot;            // partial slots per unit
  int tg;               // slots per split (FA)
  FaSplitPlan sp;       // FA only: the full-attention pass's splits (partials of item i at slots i * tg ..)
  int sa_mode;
  uint4* clear;         // 16-byte words zeroed by the kernel as a side job, or null
  int64_t n_clear;
  const float* sink;    // [Hq] sink logits (natural units of the scaled logits) or null
  const uint16_t* gate; // [B, C, Hq, D] bf16 output gate logits or null
  const float* v_scale; // [Hkv] E4M3 cache: output scale of each KV head, or null
  int hd;               // head dim (128 or 256)
};

struct PoolArgs {
  const uint16_t* q;
  const uint16_t* K;
  const int32_t* len;
  const float* stats_log2;
  float* scores;        // [rows][score_stride]
  uint32_t* hist;       // [rows][NBINS]
  const float* logits;  // [B*Hkv][C*G][logit_stride] (k_pool_logits)
  int64_t logit_stride;
  const float* k_scale;  // [Hkv] for an E4M3 cache, else null
  int hd;                // head dim (128 or 256)
  int64_t stride_b, stride_h, stride_t;
  int64_t score_stride;
  float c2;
  int B, C, Hq, Hkv, G, Gp, max_len, W;
  int split_tokens, n_split;
  int k_stream;          // k_pool: K rows are read non-temporal (the last pass over them)
};

struct SelArgs {
  const float* scores;
  const int32_t* len;
  uint32_t* hist;       // [rows][NBINS]
  int32_t* state;       // [rows][8]
  uint64_t* bitmap;     // [rows][bitmap_words]
  uint32_t* cand_key;   // [rows][cand_cap]
  int32_t* cand_idx;    // [rows][cand_cap]
  int32_t* idx;         // [rows][S]
  int64_t rows, score_stride, bitmap_words, cand_cap;
  int B, C, Hkv, max_len, k, W, S;
  int chunk;
};

struct BlockSelArgs {
  const float* scores;  // [rows][score_stride]
  const int32_t* len;
  int32_t* idx;         // [rows][S]
  uint32_t* keys;       // [rows][key_stride] block score keys (workspace)
  int64_t rows, score_stride, key_stride;
  int C, Hkv, max_len, k, W, S;
  int block;            // tokens per block, a power of two in [16, 256]; ceil(max_len / block) <= 16384
};

struct SaArgs {
  const uint16_t* q;
  const uint16_t* K;
  const uint16_t* V;
  const int32_t* len;
  const int32_t* idx;   // [B*Hkv*C][idx_stride]
  float* part_o;
  float* part_ml;
  int64_t stride_b, stride_h, stride_t, idx_stride;
  float c2;
  int B, C, Hq, Hkv, G, max_len;
  int n_slots, split_slots, n_split;
  const float* k_scale;  // [Hkv] for an E4M3 cache, else null
  int hd;                // head dim (128 or 256)
};

constexpr int kFaVariants = 9;             // full-attention kernel shapes (see HS2_RING_VARIANTS)
int fa_token_groups(int RT, int variant);  // partial slots per token split
// token groups that stream contiguous parts of one split through their own
// rings (ring kernels; merged in LDS into one partial), 1 otherwise
int fa_ring_token_groups(int RT, int variant);
int fa_split_align(int RT, int variant);   // split lengths are multiples of this many tokens
// head dim served by full-attention kernel (RT, variant) for the cache format, 0 if there is none
int fa_variant_head_dim(int RT, int variant, bool kv8);
// workgroups of the full-attention kernel (RT, variant) resident per compute
// unit on the current device (0 if that kernel does not exist)
hipError_t fa_wgs_per_cu(int RT, int variant, bool kv8, int* wgs);
hipError_t launch_fa_split(const FaArgs& a, int RT, int variant, hipStream_t s);  // a.k_scale: E4M3 cache
hipError_t launch_combine(const CombineArgs& a, int rows_per_unit, int64_t units, hipStream_t s);
hipError_t launch_pool(const PoolArgs& a, int RT, hipStream_t s);
hipError_t launch_pool_logits(const PoolArgs& a, hipStream_t s);
// workgroups of k_pool (RT, Gp, cache format, head dim) with C queries resident per compute unit
hipError_t pool_wgs_per_cu(int RT, int Gp, int C, bool kv8, int hd, int* wgs);
hipError_t set_pool_smem_limits();
hipError_t launch_sel_init(const SelArgs& a, hipStream_t s);
hipError_t launch_sel_hist(const SelArgs& a, int nchunks, hipStream_t s);
hipError_t launch_select(const SelArgs& a, hipStream_t s);
hipError_t launch_block_select(const BlockSelArgs& a, hipStream_t s);  // block sums + selection
hipError_t launch_sa_split(const SaArgs& a, int RT, hipStream_t s);
// streaming-read probe over n16 16-byte words (mode: 0 register loads, 1
// non-temporal register loads, 2 direct-to-LDS loads, 3 non-temporal
// direct-to-LDS loads); workgroup w stores a fold of its slice to sink[w]
constexpr int STREAM_PROBE_WORKGROUPS = 4096;
hipError_t launch_stream_probe(const void* src, int64_t n16, int mode, uint32_t* sink, hipStream_t s);

}  // namespace hs2
