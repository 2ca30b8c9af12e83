// HIP kernels of the hybrid-block decode path (gfx950).
//
//   k_fa_ring     full attention, split-KV flash decode through per-token-group
//                 LDS rings (bf16 or E4M3 cache, head dim 128 or 256): per
//                 (sequence, KV head, token split) a partial (m, l, O) of every
//                 query row of the group; optionally each row's logits
//   k_fa_split    the same with 64-row stages shared by 4 or 8 waves (up to
//                 128 query rows per KV head, bf16, head dim 128)
//   k_combine     merge of the partials -> bf16 output and (M, Z) per query
//                 row (sparse layers: sink logits, output gates)
//   k_pool        re-reads K, recomputes the same logits, turns them into exact
//                 probabilities with the merged (M, Z) and sums them over the
//                 query heads of the KV head -> pooled score per candidate
//                 token; builds the first-level radix histogram of the scores
//   k_pool_logits the same scores from the stored logits (few query rows)
//   k_sel_*       top-k outside the window (radix select on the score keys,
//                 ties to the lower index) + window union + ascending emission
//   k_block_*     block-level selection (block score keys, top blocks, emission)
//   k_sa_ring     sparse attention over gathered selected rows (same partial
//                 format, merged by k_combine)
//
// Query rows of one (sequence, KV head) group are laid out query-major:
// row r = c * Gp + h with Gp = G rounded up to a power of two; rows with
// h >= G or c >= C are padding (zero queries, never written out).
#include <type_traits>

#include "hs2_device.h"
#include "hs2_launch.h"

namespace hs2 {

// ============================================================================ helpers
__device__ inline int clamp_len(const int32_t* len, int b, int max_len) {
  int L = len[b];
  return L < 0 ? 0 : (L > max_len ? max_len : L);
}

// Load B operands (Q^T) of query row tile rt for this lane: row 16 rt + (lane & 15)
// (head dim 32 NKK), in the k order of q_koff.
template <int NKK>
__device__ inline void load_q_tile(uint4 (&q)[NKK], const uint16_t* __restrict__ qbase, int rt, int lane, int Gp,
                                   int G, int C, int Hq, int g, int b) {
  const int r = 16 * rt + (lane & 15);
  const int c = r / Gp, h = r % Gp;
  if (c < C && h < G) {
    const uint16_t* p = qbase + (((int64_t)b * C + c) * Hq + g * G + h) * (32 * NKK);
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) q[kk] = *(const uint4*)(p + q_koff(kk, lane));
  } else {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) q[kk] = make_uint4(0, 0, 0, 0);
  }
}

// ---------------------------------------------------------------------------- balanced token splits
// The full-attention pass cuts each sequence's cache into splits of S tokens
// and gives every (sequence, KV head, split) item one workgroup of a 1-D
// grid of sp.n_items workgroups (one residency round).  The lengths live on
// the device, so every workgroup of the pass and of its merge derives the
// same S from len[]: the shortest multiple of sp.align, at least
// sp.min_split, whose items number at most n_items -- ragged lengths then
// fill the grid evenly instead of leaving the workgroups past a short
// sequence's end idle.  sp.fixed > 0 fixes S instead (the grid then covers
// every split of the capacity).  Items are numbered sequence-major, then KV
// head, then split.  Each wave computes these wave-uniform values on its own
// (lanes over sequences), so nothing is shared or cleared between launches.
__device__ inline long long wave_sum_ll(long long v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// The clamped lengths of the sequences b = lane, lane + 64, ...: the first
// held in a register (every sequence of a batch of up to 64), the rest
// reloaded where a pass needs them.
struct LaneLens {
  const int32_t* len;
  int B, max_len, l0;
  __device__ LaneLens(const int32_t* len_, int B_, int max_len_) : len(len_), B(B_), max_len(max_len_) {
    const int lane = threadIdx.x & 63;
    l0 = lane < B ? clamp_len(len, lane, max_len) : 0;
  }
  // f(b, L) for each of this lane's sequences
  template <class F>
  __device__ void for_each(F&& f) const {
    const int lane = threadIdx.x & 63;
    if (lane < B) f(lane, l0);
    for (int b = lane + 64; b < B; b += 64) f(b, clamp_len(len, b, max_len));
  }
};

// (sequence, KV head, split) items of split length S
__device__ inline long long fa_items_of(const LaneLens& ll, int Hkv, int S) {
  long long n = 0;
  ll.for_each([&](int, int L) { n += (L + S - 1) / S; });
  return wave_sum_ll(n) * Hkv;
}

__device__ inline int fa_split_len(const LaneLens& ll, int Hkv, const FaSplitPlan& sp) {
  if (sp.fixed > 0) return sp.fixed;
  long long tot = 0;
  ll.for_each([&](int, int L) { tot += L; });
  tot = wave_sum_ll(tot) * Hkv;  // token rows over every (sequence, KV head)
  const long long units = (long long)ll.B * Hkv;
  const long long al = sp.align;
  // items(S) >= tot / S, so S >= tot / n_items; items(S) <= tot / S + units,
  // so S = tot / (n_items - units) fits (with n_items > units), as does any
  // S of at least the capacity (the host makes n_items >= units)
  const long long cap_u = (ll.max_len + al - 1) / al;
  long long lo = max((sp.min_split + al - 1) / al, (tot + sp.n_items * al - 1) / (sp.n_items * al));
  long long hi = sp.n_items > units ? (tot + (sp.n_items - units) * al - 1) / ((sp.n_items - units) * al) : cap_u;
  hi = max(min(hi, cap_u), lo);  // items(lo) <= items(hi) when hi is raised to lo
  while (lo < hi) {  // items(S) falls as S grows: the smallest S that fits
    const long long mid = (lo + hi) / 2;
    if (fa_items_of(ll, Hkv, (int)(mid * al)) <= sp.n_items)
      hi = mid;
    else
      lo = mid + 1;
  }
  return __builtin_amdgcn_readfirstlane((int)(hi * al));
}

// The (sequence, KV head, split) of item `item` with split length S; false
// if the item is past the last one (its workgroup has nothing to do).
__device__ inline bool fa_locate(const LaneLens& ll, int Hkv, int S, int item, int& b, int& g, int& split) {
  const int lane = threadIdx.x & 63;
  int rem = item;
  for (int b0 = 0; b0 < ll.B; b0 += 64) {
    const int bb = b0 + lane;
    const int L = b0 == 0 ? ll.l0 : (bb < ll.B ? clamp_len(ll.len, bb, ll.max_len) : 0);
    const int nb = (L + S - 1) / S;
    int incl = nb * Hkv;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    const unsigned long long hit = __ballot(incl > rem);
    if (hit) {
      const int l = __ffsll((long long)hit) - 1;
      const int n = __shfl(nb, l);
      const int r = rem - (__shfl(incl, l) - n * Hkv);  // item within sequence b0 + l
      b = __builtin_amdgcn_readfirstlane(b0 + l);
      g = __builtin_amdgcn_readfirstlane(r / n);
      split = __builtin_amdgcn_readfirstlane(r % n);
      return true;
    }
    rem -= __shfl(incl, 63);
  }
  return false;
}

// First item of (sequence b, KV head g) with split length S.
__device__ inline int fa_first_item(const LaneLens& ll, int Hkv, int S, int b, int g) {
  long long n = 0;
  int nb = 0;  // splits of sequence b (on the lane holding it)
  ll.for_each([&](int bb, int L) {
    if (bb < b) n += (L + S - 1) / S;
    if (bb == b) nb = (L + S - 1) / S;
  });
  n = wave_sum_ll(n) * Hkv;
  nb = __shfl(nb, b & 63);  // lane b % 64 holds sequence b
  return (int)n + g * nb;
}

// ============================================================================ full attention
// grid (items), 64 * NW threads, dynamic LDS = FA_STAGES * STAGE_BYTES.
// Cache rows stream global -> LDS with no register staging (16-byte direct
// LDS loads), FA_STAGES - 1 tiles in flight while one is computed; a single
// barrier per tile.  NW = 4 waves for up to 32 query rows, 8 above (two
// waves per SIMD).  The waves form RTW row-tile groups x TGN token groups:
// each wave owns RPW row tiles and BPW of the four 16-row blocks of a tile.
template <int RT>
struct FaShape {
  static constexpr int NW = RT >= 4 ? 8 : 4;
  static constexpr int RTW = RT < NW ? RT : NW;
  static constexpr int TGN = NW / RTW;
  static constexpr int RPW = RT / RTW;
  static constexpr int BPW = 4 / TGN;
};

template <int RT>
__global__ __launch_bounds__(512) void k_fa_split(FaArgs a) {
  using SH = FaShape<RT>;
  constexpr int NW = SH::NW, RPW = SH::RPW, BPW = SH::BPW, TG = SH::TGN, RTW = SH::RTW;
  constexpr int LPW = 16 / NW;
  extern __shared__ __align__(16) unsigned char smem[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const LaneLens ll(a.len, a.B, a.max_len);
  const int S = fa_split_len(ll, a.Hkv, a.sp);
  int b, g, split;
  if (!fa_locate(ll, a.Hkv, S, blockIdx.x, b, g, split)) return;
  const int Lv = clamp_len(a.len, b, a.max_len);
  const int t_begin = split * S;
  const int t_end = min(Lv, t_begin + S);
  const int ntiles = (t_end - t_begin + TILE - 1) / TILE;
  const int tg = wave / RTW;
  const int rt0 = (wave % RTW) * RPW;

  uint4 q[RPW][4];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) load_q_tile(q[rr], a.q, rt0 + rr, lane, a.Gp, a.G, a.C, a.Hq, g, b);
  // causal position of each of this lane's query rows (padding rows see everything)
  int rpos[RPW];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    const int c = (16 * (rt0 + rr) + (lane & 15)) / a.Gp;
    rpos[rr] = c < a.C ? Lv - a.C + c : Lv - 1;
  }
  const int min_pos = Lv - a.C;

  const int64_t kvoff = (int64_t)b * a.stride_b + (int64_t)g * a.stride_h;
  const uint16_t* Kbg = a.K + kvoff;
  const uint16_t* Vbg = a.V + kvoff;

  auto issue = [&](int tile) {
    const int t0 = t_begin + tile * TILE;
    int tok[LPW];
#pragma unroll
    for (int u = 0; u < LPW; ++u) {
      const int t = t0 + stage_row<NW>(wave, u, lane);
      tok[u] = t < t_end ? t : t_end - 1;  // rows past the range repeat a valid row; masked below
    }
    issue_stage_loads<NW>(smem + (tile % FA_STAGES) * STAGE_BYTES, Kbg, Vbg, a.stride_t, tok, wave, lane);
  };

  WaveState<RPW> st;
  st.init();
  int blk[BPW];
#pragma unroll
  for (int bi = 0; bi < BPW; ++bi) blk[bi] = tg * BPW + bi;

#pragma unroll
  for (int i = 0; i < FA_STAGES - 1; ++i)
    if (i < ntiles) issue(i);
  for (int i = 0; i < ntiles; ++i) {
    // stages issued after tile i by this wave: min(FA_STAGES - 2, ntiles - 1 - i)
    wait_stage_loads<NW>(min(FA_STAGES - 2, ntiles - 1 - i));
    __syncthreads();
    if (i + FA_STAGES - 1 < ntiles) issue(i + FA_STAGES - 1);
    const unsigned char* stg = smem + (i % FA_STAGES) * STAGE_BYTES;
    const int t0 = t_begin + i * TILE;
    f32x4 S[BPW][RPW];
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) qk_block_swz<RPW>(stg, blk[bi], q, S[bi], lane);
    const bool full = (t0 + TILE <= t_end) && (t0 + TILE - 1 <= min_pos);
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi)
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          float v = S[bi][rr][ii] * a.c2;
          if (!full) {
            const int t = t0 + 16 * blk[bi] + 4 * (lane >> 4) + ii;
            if (t >= t_end || t > rpos[rr]) v = -INFINITY;
          }
          S[bi][rr][ii] = v;
        }
    softmax_pv_swz<RPW, BPW>(st, stg, blk, S, lane);
  }
  const int64_t slot_base_row = ((int64_t)blockIdx.x * TG + tg) * (16 * RT);
  store_partial<RPW>(st, a.part_o, a.part_ml, slot_base_row, rt0, lane);
}

// ---------------------------------------------------------------------------- ring variant
// grid (n_split, Hkv, B), 64 * NWV threads (NWV = 1 or 2 waves), dynamic LDS
// = NS stages of TW rows of K and V.  The workgroup owns a contiguous token
// split of one (b, g); each wave owns RT / NWV query row tiles.  The split
// streams through a private ring with NS - 1 stages in flight; with one wave
// there is no barrier at all, with two waves one barrier per stage.  One
// partial (m, l, O) per split.
// KV8: the cache is E4M3 bytes with one scale per KV head (k_scale folds
// into the logit scale, v_scale is applied by the merge); each token group
// stages raw rows in its ring (swizzled by raw_swz).  A one-wave group reads
// the K operands raw and the V operands raw by 8-bit transposing LDS reads,
// both converted in registers (no tile, no barrier); a group of several
// waves converts each tile's K and V rows once into shared bf16 tiles (one
// barrier per tile), which its waves read as the bf16 path reads its stage
// (each wave converting the whole tile itself measured 1.45x slower at 64
// query rows per KV head).  HDIM: head dim (128 or 256).  KP: cache policy
// of the stage loads (FaCachePolicy).
template <int RT, int NWV, int TW, int NS, int TGW, bool KV8, int HDIM, int KP>
__global__ __launch_bounds__(64 * NWV * TGW) void k_fa_ring(FaArgs a) {
  constexpr int RPW = RT / NWV;
  constexpr int NB = TW / 16;                              // 16-row blocks per stage
  constexpr int NKK = HDIM / 32;                           // 32-wide k steps of the logits
  constexpr int SRB = 2 * HDIM;                            // bytes of a bf16 stage row
  constexpr int RB = KV8 ? HDIM : SRB;                     // bytes of a staged cache row
  constexpr int CPR = RB / 16;                             // 16-byte chunks per staged row
  constexpr int LPM = TW * RB / 1024 / NWV;                // 1 KB loads per matrix per stage per wave
  constexpr int SB = 2 * TW * RB;                          // ring stage: K rows then V rows
  constexpr int GB = fa_ring_group_bytes(NWV, TW, NS, KV8, HDIM);  // LDS of one token group: ring + tiles
  // E4M3 with several waves per group: K and V are converted once into
  // shared bf16 tiles (each wave would otherwise convert the whole tile for
  // its own row tiles)
  constexpr bool KCONV = KV8 && NWV > 1;
  static_assert(LPM >= 1 && TW * RB == 1024 * LPM * NWV, "whole 1 KB loads for every wave and stage");
  static_assert(TGW == 1 || RT > 1, "token groups are not combined with the logits output");
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int tg = wid / NWV, wave = wid % NWV;  // token group, wave in it
  const LaneLens ll(a.len, a.B, a.max_len);
  const int S = __builtin_amdgcn_readfirstlane(fa_split_len(ll, a.Hkv, a.sp));
  int b, g, split;
  if (!fa_locate(ll, a.Hkv, S, blockIdx.x, b, g, split)) return;
  // uniform by construction; said so, so that every address derived from
  // them stays in scalar registers
  b = __builtin_amdgcn_readfirstlane(b);
  g = __builtin_amdgcn_readfirstlane(g);
  split = __builtin_amdgcn_readfirstlane(split);
  const int Lv = __builtin_amdgcn_readfirstlane(clamp_len(a.len, b, a.max_len));
  // token group tg streams the tg-th contiguous part of the split through its own ring
  const int part = S / TGW;
  const int t_begin = split * S + tg * part;
  const int t_end = min(Lv, t_begin + part);
  const int ntiles = t_end > t_begin ? (t_end - t_begin + TW - 1) / TW : 0;
  const int nloop = (min(Lv, split * S + part) - split * S + TW - 1) / TW;  // group 0's
  // a located item's split starts below the length, so group 0 has a tile:
  // without a zero-trip path the accumulators leave the loop in their own
  // registers (with it the compiler copied all of O at every tile)
  __builtin_assume(nloop >= 1);
  // FA_STREAM_K_HEAD: K rows of the group before this offset are non-temporal
  const int k_stream = part - (int)((int64_t)part * a.k_keep_pct / 100);
  const int rt0 = wave * RPW;

  uint4 q[RPW][NKK];
  int rpos[RPW];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    load_q_tile(q[rr], a.q, rt0 + rr, lane, a.Gp, a.G, a.C, a.Hq, g, b);
    const int c = (16 * (rt0 + rr) + (lane & 15)) / a.Gp;
    rpos[rr] = c < a.C ? Lv - a.C + c : Lv - 1;  // padding rows see everything
  }
  const int min_pos = Lv - a.C;
  constexpr int ESZ = KV8 ? 1 : 2;  // bytes per cache element
  const int64_t kvoff = ((int64_t)b * a.stride_b + (int64_t)g * a.stride_h) * ESZ;
  const unsigned char* Kbg = (const unsigned char*)a.K + kvoff;
  const unsigned char* Vbg = (const unsigned char*)a.V + kvoff;
  const int64_t stride_t = a.stride_t * ESZ;  // bytes
  const float c2 = KV8 ? a.c2 * a.k_scale[g] : a.c2;
  const uint32_t ring = lds_addr(smem) + (uint32_t)(tg * GB);
  unsigned char* ring_p = smem + tg * GB;
  unsigned char* tile_k = ring_p + NS * SB;   // KCONV: the converted K tile
  unsigned char* tile_v = tile_k + TW * SRB;  // KCONV: the converted V tile
  // logits output of a single row tile (C G <= 16 query rows): this lane's
  // row (c, h), or null.  Row-major [B*Hkv][C*G][logit_stride], log2 units.
  float* lrow = nullptr;
  if constexpr (RT == 1) {
    const int r = lane & 15;
    const int c = r / a.Gp, h = r % a.Gp;
    if (a.logits && c < a.C && h < a.G)
      lrow = a.logits + (((int64_t)b * a.Hkv + g) * a.C * a.G + c * a.G + h) * a.logit_stride;
  }

  // per-lane part of each load's byte offset from its tile's first row (32
  // bits: a tile spans TW rows, and the host keeps TW token strides below
  // 2^31 bytes): a 1 KB load covers RPL rows of CPR chunks (lane / CPR =
  // row, lane % CPR = chunk slot); bf16 rows are swizzled, E4M3 rows raw.
  // The tile's first row is a wave-uniform base in scalar registers.
  constexpr int RPL = 1024 / RB;  // rows per 1 KB load
  auto lane_offset = [&](int row, int dt) -> uint32_t {
    return (uint32_t)(dt * (int)stride_t) +
           16u * (uint32_t)((lane % CPR) ^ (KV8 ? raw_swz<RB>(row) : stage_swz(row)));
  };
  uint32_t lane_off[LPM];
#pragma unroll
  for (int u = 0; u < LPM; ++u) {
    const int row = RPL * (wave * LPM + u) + lane / CPR;
    lane_off[u] = lane_offset(row, row);
  }
  // K_NT: this tile's K rows are loaded non-temporal (V rows: every policy
  // but the default)
  auto issue_as = [&](int tile, auto k_nt) __attribute__((always_inline)) {
    const int t0 = t_begin + tile * TW;
    const uint32_t base = ring + (uint32_t)((tile % NS) * SB);
    const bool whole = t0 + TW <= t_end;
    const unsigned char* kt = Kbg + (int64_t)t0 * stride_t;
    const unsigned char* vt = Vbg + (int64_t)t0 * stride_t;
#pragma unroll
    for (int u = 0; u < LPM; ++u) {
      const int n = wave * LPM + u;
      uint32_t off = lane_off[u];
      if (!whole) {  // rows past the range repeat the last valid row; masked below
        const int row = RPL * n + lane / CPR;
        off = lane_offset(row, min(t0 + row, t_end - 1) - t0);
      }
      dma16_s<decltype(k_nt)::value>(kt, off, __builtin_amdgcn_readfirstlane(base + 1024 * n));
      dma16_s<KP != FA_CACHE_DEFAULT>(vt, off, __builtin_amdgcn_readfirstlane(base + TW * RB + 1024 * n));
    }
  };
  auto issue = [&](int tile) __attribute__((always_inline)) {
    if constexpr (KP == FA_STREAM_K_HEAD) {  // one scalar branch per tile
      if (tile * TW < k_stream)
        issue_as(tile, std::true_type{});
      else
        issue_as(tile, std::false_type{});
    } else {
      issue_as(tile, std::integral_constant<bool, KP == FA_STREAM_KV>{});
    }
  };

  WaveState<RPW, HDIM> st;
  st.init();
#pragma unroll
  for (int i = 0; i < NS - 1; ++i)
    if (i < ntiles) issue(i);
  // every wave runs group 0's tile count of barrier rounds (the counts must
  // match): its own tiles here, then barrier-only rounds for the rest (a
  // loop of its own, so that the tile loop has no path that leaves the
  // accumulators untouched: with one, the compiler copied all of O into a
  // second register set at every tile)
  for (int i = 0; i < ntiles; ++i) {
    // logits stores also count in vmcnt; they only make this wait longer
    wait_ring<2 * LPM>(min(NS - 2, ntiles - 1 - i));
    if (NWV * TGW > 1) __syncthreads();
    if (i + NS - 1 < ntiles) issue(i + NS - 1);
    const unsigned char* stg = ring_p + (i % NS) * SB;
    if constexpr (KCONV) {
      convert_rows_e4m3<TW, 64 * NWV, HDIM>(stg, tile_k, 64 * wave + lane);
      convert_rows_e4m3<TW, 64 * NWV, HDIM>(stg + TW * RB, tile_v, 64 * wave + lane);
      __syncthreads();  // both tiles converted by every wave of the group
    }
    const int t0 = t_begin + i * TW;
    f32x4 S[NB][RPW];
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      if constexpr (KCONV)
        qk_block_swz<RPW>(tile_k, bi, q, S[bi], lane);
      else if constexpr (KV8)
        qk_block_e4m3<RPW, RB>(stg, bi, q, S[bi], lane);
      else
        qk_block_swz<RPW>(stg, bi, q, S[bi], lane);
    }
    if constexpr (RT == 1) {  // the lane's 4 consecutive tokens; the row stride covers whole tiles
      if (lrow)
#pragma unroll
        for (int bi = 0; bi < NB; ++bi) *(f32x4*)(lrow + t0 + 16 * bi + 4 * (lane >> 4)) = S[bi][0] * c2;
    }
    const bool full = (t0 + TW <= t_end) && (t0 + TW - 1 <= min_pos);
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          float v = S[bi][rr][ii] * c2;
          if (!full) {
            const int t = t0 + 16 * bi + 4 * (lane >> 4) + ii;
            if (t >= t_end || t > rpos[rr]) v = -INFINITY;
          }
          S[bi][rr][ii] = v;
        }
    PFrags<NB, RPW> pf;
    online_softmax(st, S, pf, lane);
    if constexpr (KCONV)
      pv_tile<RPW, NB, HDIM>(st, pf, tile_v, lane);
    else if constexpr (KV8)  // V read raw (transposing 8-bit reads) and converted in registers
      pv_tile_e4m3<RPW, NB, HDIM, RB>(st, pf, stg + TW * RB, lane);
    else
      pv_tile<RPW, NB, HDIM>(st, pf, stg + TW * SRB, lane);
  }
  for (int i = ntiles; i < nloop; ++i) {  // a group past its own tiles: group 0's barriers
    if (NWV * TGW > 1) __syncthreads();
    if (KCONV) __syncthreads();  // its K-tile barrier
  }
  const int64_t slot_base_row = (int64_t)blockIdx.x * (16 * RT);  // one partial per item
  if constexpr (TGW == 1) {
    store_partial<RPW>(st, a.part_o, a.part_ml, slot_base_row, rt0, lane);
  } else {
    // merge the token groups in LDS (the rings are free), one partial per split
    constexpr int ROWS = 16 * RT;
    __syncthreads();
    float* mlL = (float*)smem;              // [TGW][ROWS][4]: (m ref, l, m true, -)
    float* oL = mlL + TGW * ROWS * 4;       // [TGW - 1][ROWS][HDIM]: the other groups' O
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
      const float l = sum_xor32(sum_xor16(st.l[rr]));
      const int row0 = 16 * (rt0 + rr);
      if (lane < 16) *(float4*)(mlL + (tg * ROWS + row0 + lane) * 4) = make_float4(st.m[rr], l, st.mt[rr], 0.f);
      if (tg > 0)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int nb = 0; nb < HDIM / 16; ++nb)
            oL[((tg - 1) * ROWS + row0 + 4 * (lane >> 4) + i) * HDIM + 16 * nb + (lane & 15)] = st.o[rr][nb][i];
    }
    __syncthreads();
    if (tg > 0) return;
    // weight of group j's row R against the rows' common maximum (a group
    // without tokens has m = -inf and weight 0)
    auto weights = [&](int R, float (&f)[TGW], float& M) {
      M = -INFINITY;
#pragma unroll
      for (int j = 0; j < TGW; ++j) M = fmaxf(M, mlL[(j * ROWS + R) * 4]);
#pragma unroll
      for (int j = 0; j < TGW; ++j) {
        const float m = mlL[(j * ROWS + R) * 4];
        f[j] = m == -INFINITY ? 0.f : fast_exp2(m - M);
      }
    };
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
      const int row0 = 16 * (rt0 + rr);
      if (lane < 16) {
        float f[TGW], M;
        weights(row0 + lane, f, M);
        float l = 0.f, mt = -INFINITY;
#pragma unroll
        for (int j = 0; j < TGW; ++j) {
          l += mlL[(j * ROWS + row0 + lane) * 4 + 1] * f[j];
          mt = fmaxf(mt, mlL[(j * ROWS + row0 + lane) * 4 + 2]);
        }
        *(float4*)(a.part_ml + (slot_base_row + row0 + lane) * 4) = make_float4(M, l, mt, 0.f);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int R = row0 + 4 * (lane >> 4) + i;
        float f[TGW], M;
        weights(R, f, M);
        float* dst = a.part_o + (slot_base_row + R) * HDIM + (lane & 15);
#pragma unroll
        for (int nb = 0; nb < HDIM / 16; ++nb) {
          float o = st.o[rr][nb][i] * f[0];
#pragma unroll
          for (int j = 1; j < TGW; ++j) o += oL[((j - 1) * ROWS + R) * HDIM + 16 * nb + (lane & 15)] * f[j];
          dst[16 * nb] = o;
        }
      }
    }
  }
}

// ============================================================================ combine
// grid (rows_per_unit, units), 256 threads = 256 / NQ slot groups x NQ =
// HDIM / 4 column quads.
// FA: unit = (b, g), row r = c * Gp + h; slots valid = ceil(Lv / split) * TG.
// SA: unit = (b, g, c), row = h; all n_split * TG slots written.
template <int HDIM>
__global__ __launch_bounds__(256) void k_combine(CombineArgs a) {
  constexpr int NQ = HDIM / 4, SG = 256 / NQ;
  __shared__ float s_m[SG], s_mt[SG], s_z[SG];
  __shared__ float4 s_o[SG][NQ];
  const int r = blockIdx.x;
  const int64_t unit = blockIdx.y;
  const int tid = threadIdx.x;
  const int sg = tid / NQ, dq = tid % NQ;
  if (a.clear) {  // zero the selection histogram and counters for the kernels that follow
    const int64_t nb = (int64_t)gridDim.x * gridDim.y, bid = unit * gridDim.x + r;
    for (int64_t i = bid * 256 + tid; i < a.n_clear; i += nb * 256) a.clear[i] = make_uint4(0, 0, 0, 0);
  }
  int b, g, c, h;
  if (a.sa_mode) {
    c = (int)(unit % a.C);
    g = (int)((unit / a.C) % a.Hkv);
    b = (int)(unit / ((int64_t)a.C * a.Hkv));
    h = r;
  } else {
    g = (int)(unit % a.Hkv);
    b = (int)(unit / a.Hkv);
    c = r / a.Gp;
    h = r % a.Gp;
  }
  if (c >= a.C || h >= a.G) return;
  int nvalid = a.nslot;
  int64_t base = unit * a.nslot * a.rows + r;
  if (!a.sa_mode) {  // the full-attention items of (b, g): their slots are contiguous
    const LaneLens ll(a.len, a.B, a.max_len);
    const int S = fa_split_len(ll, a.Hkv, a.sp);
    const int Lv = clamp_len(a.len, b, a.max_len);
    nvalid = ((Lv + S - 1) / S) * a.tg;
    base = (int64_t)fa_first_item(ll, a.Hkv, S, b, g) * a.tg * a.rows + r;
  }
  // one pass over the partials: each slot group merges its slots online
  // (reference maximum m, sum l, output row, rescaled when m rises) with
  // every slot's loads issued together, then the groups are merged in LDS
  float m = -INFINITY, mt = -INFINITY, z = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int s = sg; s < nvalid; s += SG) {
    const int64_t pr = base + (int64_t)s * a.rows;
    const float4 ml = *(const float4*)(a.part_ml + pr * 4);
    const float4 o = *(const float4*)(a.part_o + pr * HDIM + 4 * dq);
    mt = fmaxf(mt, ml.z);
    const float mn = fmaxf(m, ml.x);
    // an empty partial (m = -inf, O = 0) adds nothing; exp2(-inf) = 0
    const float keep = mn == -INFINITY ? 1.f : fast_exp2(m - mn);
    const float w = mn == -INFINITY ? 0.f : fast_exp2(ml.x - mn);
    z = z * keep + ml.y * w;
    acc.x = acc.x * keep + o.x * w;
    acc.y = acc.y * keep + o.y * w;
    acc.z = acc.z * keep + o.z * w;
    acc.w = acc.w * keep + o.w * w;
    m = mn;
  }
  if (dq == 0) {
    s_m[sg] = m;
    s_mt[sg] = mt;
  }
  __syncthreads();
  float M = -INFINITY, Mt = -INFINITY;
#pragma unroll
  for (int j = 0; j < SG; ++j) {
    M = fmaxf(M, s_m[j]);
    Mt = fmaxf(Mt, s_mt[j]);
  }
  const int64_t orow = ((int64_t)b * a.C + c) * a.Hq + (int64_t)g * a.G + h;
  // sink logit of this head in log2 units: joins the normaliser, no value row
  const float sink2 = a.sink ? a.sink[g * a.G + h] * 1.4426950408889634f : -INFINITY;
  M = fmaxf(M, sink2);
  const float f = M == -INFINITY ? 0.f : fast_exp2(m - M);  // this group's share
  s_o[sg][dq] = make_float4(acc.x * f, acc.y * f, acc.z * f, acc.w * f);
  if (dq == 0) s_z[sg] = z * f;
  __syncthreads();
  if (sg != 0) return;
  float Z = 0.f;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < SG; ++j) {
    Z += s_z[j];
    o.x += s_o[j][dq].x;
    o.y += s_o[j][dq].y;
    o.z += s_o[j][dq].z;
    o.w += s_o[j][dq].w;
  }
  if (sink2 != -INFINITY) Z += fast_exp2(sink2 - M);
  const float inv = (Z > 0.f ? 1.f / Z : 0.f) * (a.v_scale ? a.v_scale[g] : 1.f);
  o.x *= inv;
  o.y *= inv;
  o.z *= inv;
  o.w *= inv;
  if (a.gate) {  // out *= sigmoid(gate), elementwise
    const uint2 gb = *(const uint2*)(a.gate + orow * HDIM + 4 * dq);
    const float gv[4] = {bf16_bits_to_f32(gb.x & 0xFFFFu), bf16_bits_to_f32(gb.x >> 16), bf16_bits_to_f32(gb.y & 0xFFFFu),
                         bf16_bits_to_f32(gb.y >> 16)};
    float gsig[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) gsig[j] = 1.f / (1.f + fast_exp2(-gv[j] * 1.4426950408889634f));
    o.x *= gsig[0];
    o.y *= gsig[1];
    o.z *= gsig[2];
    o.w *= gsig[3];
  }
  uint2 packed;
  packed.x = f32_to_bf16_bits(o.x) | (f32_to_bf16_bits(o.y) << 16);
  packed.y = f32_to_bf16_bits(o.z) | (f32_to_bf16_bits(o.w) << 16);
  *(uint2*)(a.out + orow * HDIM + 4 * dq) = packed;
  if (dq == 0) {
    if (a.stats_log2) {
      a.stats_log2[orow * 2] = M;
      a.stats_log2[orow * 2 + 1] = Z;
    }
    if (a.stats_user) {  // against the true maximum: Z * 2^(M - Mt), M <= Mt
      a.stats_user[orow * 2] = Mt == -INFINITY ? Mt : Mt * 0.69314718055994531f;
      a.stats_user[orow * 2 + 1] = Mt == -INFINITY ? 0.f : Z * fast_exp2(M - Mt);
    }
  }
}

// ============================================================================ pooled scores
// Token scores of the full-attention layer: for query c and candidate token t,
// P = sum over the heads h of query c of exp2(s2_h(t) - M2_h) / Z_h, with the
// same logits s2 the full-attention kernel used and its merged (M2, Z).
//
// Both score kernels write every candidate's score and the rows' first-level
// histogram of score keys: k_pool recomputes the logits from K, k_pool_logits
// reads the ones the full-attention kernel stored.  Logits are computed as
// S = Q . K^T (query rows on MFMA rows), so lane l holds rows 4(l/16)+i of
// token l%16: the GP heads of a query are summed inside the lane and across
// at most two lane groups, and the 16 scores of a block sit in 16
// consecutive lanes.

// Scores of one 16-token block from the logits in acc (S = Q.K^T: lane l
// holds rows 16 (rt0 + rr) + 4 (l / 16) + i of token l % 16): p = exp2(s2 -
// msub) * fac per head, summed over the GP heads of each query (in-lane, then
// across lane groups / row tiles); emit(v, c, t) is called by the lanes
// holding query c's score of token t.
template <int RPW, int GP, class Emit>
__device__ __forceinline__ void pool_emit_block(const f32x4 (&acc)[RPW], float c2, const float (&fac)[RPW][4],
                                                const float (&msub)[RPW][4], int rt0, int t, int lane, Emit& emit) {
  const int q4 = lane >> 4;
  float e[RPW][4];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
    for (int i = 0; i < 4; ++i) e[rr][i] = fast_exp2(acc[rr][i] * c2 - msub[rr][i]) * fac[rr][i];
  if constexpr (GP == 1) {
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
      for (int i = 0; i < 4; ++i) emit(e[rr][i], 16 * (rt0 + rr) + 4 * q4 + i, t);
  } else if constexpr (GP == 2) {
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
      emit(e[rr][0] + e[rr][1], 8 * (rt0 + rr) + 2 * q4, t);
      emit(e[rr][2] + e[rr][3], 8 * (rt0 + rr) + 2 * q4 + 1, t);
    }
  } else if constexpr (GP <= 16) {
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
      float v = (e[rr][0] + e[rr][1]) + (e[rr][2] + e[rr][3]);
      if constexpr (GP >= 8) v = sum_xor16(v);
      if constexpr (GP >= 16) v = sum_xor32(v);
      // rows 16 rt + 4 q4 .. belong to query (16 rt + 4 q4) / GP; one lane group per query emits
      if (((4 * q4) & (GP - 1)) == 0) emit(v, (16 * (rt0 + rr) + 4 * q4) / GP, t);
    }
  } else if constexpr (RPW % (GP / 16) == 0) {
    constexpr int TPQ = GP / 16;  // row tiles per query, all in this wave
#pragma unroll
    for (int cq = 0; cq < RPW / TPQ; ++cq) {
      float v = 0.f;
#pragma unroll
      for (int j = 0; j < TPQ; ++j) {
        const int rr = cq * TPQ + j;
        v += (e[rr][0] + e[rr][1]) + (e[rr][2] + e[rr][3]);
      }
      v = sum_xor32(sum_xor16(v));
      if (q4 == 0) emit(v, (16 * rt0) / GP + cq, t);
    }
  } else {  // this wave holds RPW of the query's row tiles: emit its part of the sum
    static_assert((GP / 16) % RPW == 0, "a query's row tiles split evenly over its waves");
    float v = 0.f;
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) v += (e[rr][0] + e[rr][1]) + (e[rr][2] + e[rr][3]);
    v = sum_xor32(sum_xor16(v));
    if (q4 == 0) emit(v, (16 * rt0) / GP, t);
  }
}

// Scores of two 16-token blocks a and b of a one-row-tile wave (queries of
// 8 or 16 heads; acc as in pool_emit_block), packed into one register: the
// lane swap meets the odd lane groups of a with the even groups of b, so
// lane group j ends up with the sum over its rows' pair of groups for block
// j & 1 -- the same values, summed in the same order, as pool_emit_block.
template <int GP>
__device__ __forceinline__ float pool_pair_value(const f32x4& a, const f32x4& b, float c2, const float (&fac)[4],
                                                 const float (&msub)[4]) {
  float ea[4], eb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ea[i] = fast_exp2(a[i] * c2 - msub[i]) * fac[i];
    eb[i] = fast_exp2(b[i] * c2 - msub[i]) * fac[i];
  }
  const float sa = (ea[0] + ea[1]) + (ea[2] + ea[3]);
  const float sb = (eb[0] + eb[1]) + (eb[2] + eb[3]);
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(sa), __float_as_uint(sb), false, false);
  float v = __uint_as_float(r[0]) + __uint_as_float(r[1]);  // group j: block j & 1, rows of groups j & 2, (j & 2) + 1
  if constexpr (GP == 16) v = sum_xor32(v);                // and of groups j ^ 2
  return v;
}

// Row constants of rows 16 (rt0 + rr) + 4 (lane / 16) + i: p = exp2(s2 -
// msub) * fac = exp2(s2 - M2) / Z (fac = exp2(-M2) / Z unless M2 is too large
// for that, then msub = M2 and fac = 1 / Z).  Branch-free on purpose:
// conditional stores into the arrays make the compiler carry them whole.
template <int RPW, int GP>
__device__ __forceinline__ void pool_row_consts(const PoolArgs& a, int b, int g, int rt0, int lane,
                                                float (&fac)[RPW][4], float (&msub)[RPW][4]) {
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 16 * (rt0 + rr) + 4 * (lane >> 4) + i;
      const int c = r / GP, h = r % GP;
      const bool valid = c < a.C && h < a.G;  // padding rows contribute nothing
      const int64_t orow = valid ? ((int64_t)b * a.C + c) * a.Hq + (int64_t)g * a.G + h : 0;
      const float2 mz = *(const float2*)(a.stats_log2 + orow * 2);
      const float z = valid ? mz.y : 0.f;
      const bool big = !(fabsf(mz.x) < 64.f);
      const float inv_z = 1.f / z;
      fac[rr][i] = z > 0.f ? (big ? inv_z : fast_exp2(-mz.x) * inv_z) : 0.f;
      msub[rr][i] = (z > 0.f && big) ? mz.x : 0.f;
    }
}

// Scores by a second pass over K, streamed like the full-attention kernel:
// grid (token splits, Hkv, B), 64 * NWV threads; K tiles of TW tokens go
// global -> LDS through an NS-stage ring (16-byte direct loads, swizzled
// rows), every wave reads the whole tile as the MFMA B operand against its
// own query row tiles held in registers.  Dynamic LDS: ring + C packed
// first-level histograms (16-bit counters; a split has < 65536 tokens).
// KV8: E4M3 cache with one K scale per KV head (folded into the logit
// scale); raw rows are staged (swizzled by raw_swz) and each wave converts
// its K operands in registers.  HDIM: head dim (128 or 256).
template <int RT, int GP, bool KV8, int HDIM>
struct PoolShape {
  static constexpr int TPQ = GP > 16 ? GP / 16 : 1;           // row tiles per query
  // row tiles per wave: one tile per wave for queries of at most 16 heads
  // (more waves share each staged tile: 134 -> 126 us at 64 rows per KV
  // head); a query of 32 heads in one wave (its heads summed in registers);
  // of 64 heads, with a bf16 cache, in two waves whose per-token sums meet
  // in LDS (MQA 64/1: 106 -> 104 us at one query, 62 -> 54 us at two; with
  // E4M3 one wave stays 8 % faster)
  static constexpr int RPW = RT == 1 ? 1 : (TPQ > 2 && !KV8 ? TPQ / 2 : TPQ);
  static constexpr int WPQ = TPQ / RPW > 1 ? TPQ / RPW : 1;  // waves per query
  static constexpr int NWV = RT / RPW;
  static constexpr int SRB = 2 * HDIM;                        // bytes of a bf16 stage row
  static constexpr int RB = KV8 ? HDIM : SRB;                 // bytes of a staged row
  static constexpr int RPL = 1024 / RB;                       // rows per 1 KB load
  // whole 1 KB loads for every wave: at least 32 rows (bf16) or 16 (E4M3;
  // 32 made the MQA 64/1 head-dim-256 pass 14 % slower, while bf16 gained
  // 4 % at 64 rows per KV head), RPL NWV when more
  static constexpr int TW_MIN = KV8 ? 16 : 32;
  static constexpr int TW = RPL * NWV > TW_MIN ? RPL * NWV : TW_MIN;
  // 3 stages; 2 for a bf16 cache of head dim 256 (16 KB stages: one more
  // workgroup per CU, the MQA 64/1 pass 85 -> 83 us; at head dim 128 two
  // stages lose 94 -> 105 us)
  static constexpr int NS = !KV8 && HDIM == 256 ? 2 : 3;
  static constexpr int SB = TW * RB;                          // ring stage
  // E4M3 with several waves: K converted once into a shared bf16 tile
  static constexpr bool KCONV = KV8 && NWV > 1;
  // one row tile per wave of queries of 8 or 16 heads: two blocks' scores
  // are packed into the four lane groups and emitted together
  static constexpr bool PACK2 = WPQ == 1 && RPW == 1 && (GP == 8 || GP == 16) && (TW / 16) % 2 == 0;
  static constexpr int LDS = NS * SB + (KCONV ? TW * SRB : 0);  // before the histograms
};
template <int RT, int GP, bool KV8, int HDIM>
__global__ __attribute__((amdgpu_flat_work_group_size(64, 64 * PoolShape<RT, GP, KV8, HDIM>::NWV))) void k_pool(PoolArgs a) {
  using PS = PoolShape<RT, GP, KV8, HDIM>;
  constexpr int RPW = PS::RPW, NWV = PS::NWV, TW = PS::TW, NS = PS::NS, SB = PS::SB, RB = PS::RB, SRB = PS::SRB;
  constexpr int NB = TW / 16;
  constexpr int NKK = HDIM / 32;
  constexpr int CPR = RB / 16;               // 16-byte chunks per staged row
  constexpr int LPM = TW * RB / 1024 / NWV;  // 1 KB loads per stage per wave
  static_assert(LPM >= 1 && TW * RB == 1024 * LPM * NWV, "whole 1 KB loads per wave and stage");
  extern __shared__ __align__(16) unsigned char smem[];
  uint32_t* hist = (uint32_t*)(smem + PS::LDS);       // [C][NBINS/2]

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int Lv = __builtin_amdgcn_readfirstlane(clamp_len(a.len, b, a.max_len));
  // candidates of query c: [0, Lv - C + c - W + 1); their union ends at Lv - W
  const int n_cand_max = Lv - a.W;
  const int t_begin = split * a.split_tokens;
  if (t_begin >= n_cand_max) return;
  const int t_end = min(n_cand_max, t_begin + a.split_tokens);
  const int ntiles = (t_end - t_begin + TW - 1) / TW;
  const int rt0 = wave * RPW;

  for (int i = tid; i < a.C * (NBINS / 2); i += 64 * NWV) hist[i] = 0;
  uint4 q[RPW][NKK];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) load_q_tile(q[rr], a.q, rt0 + rr, lane, GP, a.G, a.C, a.Hq, g, b);
  float fac[RPW][4], msub[RPW][4];
  pool_row_consts<RPW, GP>(a, b, g, rt0, lane, fac, msub);

  constexpr int ESZ = KV8 ? 1 : 2;  // bytes per cache element
  const unsigned char* Kbg = (const unsigned char*)a.K + ((int64_t)b * a.stride_b + (int64_t)g * a.stride_h) * ESZ;
  const int64_t stride_t = a.stride_t * ESZ;
  const float c2 = KV8 ? a.c2 * a.k_scale[g] : a.c2;
  const uint32_t ring = lds_addr(smem);
  constexpr int RPL = PS::RPL;  // rows per 1 KB load
  // per-lane offsets from the tile's first row, as in the full-attention ring
  auto lane_offset = [&](int row, int dt) -> uint32_t {
    return (uint32_t)(dt * (int)stride_t) +
           16u * (uint32_t)((lane % CPR) ^ (KV8 ? raw_swz<RB>(row) : stage_swz(row)));
  };
  uint32_t lane_off[LPM];
#pragma unroll
  for (int u = 0; u < LPM; ++u) {
    const int row = RPL * (wave * LPM + u) + lane / CPR;
    lane_off[u] = lane_offset(row, row);
  }
  // tiles from the end of the split backwards: at equal split lengths the
  // full-attention pass read those rows last (2 % faster at 64 rows per KV
  // head, where the two passes' ranges coincide)
  // the last pass over these K rows: a cache larger than the last-level
  // cache streams them (non-temporal) past the caches
  auto issue_as = [&](int tile, auto k_nt) __attribute__((always_inline)) {
    const int t0 = t_begin + (ntiles - 1 - tile) * TW;
    const uint32_t base = ring + (uint32_t)((tile % NS) * SB);
    const bool whole = t0 + TW <= t_end;
    const unsigned char* kt = Kbg + (int64_t)t0 * stride_t;
#pragma unroll
    for (int u = 0; u < LPM; ++u) {
      const int n = wave * LPM + u;
      uint32_t off = lane_off[u];
      if (!whole) {  // rows past the range repeat the last valid row; never emitted
        const int row = RPL * n + lane / CPR;
        off = lane_offset(row, min(t0 + row, t_end - 1) - t0);
      }
      dma16_s<decltype(k_nt)::value>(kt, off, __builtin_amdgcn_readfirstlane(base + 1024 * n));
    }
  };
  auto issue = [&](int tile) __attribute__((always_inline)) {  // one scalar branch per tile
    if (a.k_stream)
      issue_as(tile, std::true_type{});
    else
      issue_as(tile, std::false_type{});
  };
  __syncthreads();  // histogram cleared before any wave adds to it

  float* scores = a.scores + ((int64_t)b * a.Hkv + g) * a.C * a.score_stride;
  const int nc0 = Lv - a.C - a.W + 1;  // candidates of query 0 (query c: nc0 + c)
  int t0_tile = 0;
  __shared__ float s_part[PS::WPQ > 1 ? NWV * TW : 1];  // per-token parts of split queries
  auto emit_part = [&](float v, int, int t) { s_part[wave * TW + (t - t0_tile)] = v; };
  auto emit = [&](float v, int c, int t) {
    if (c < a.C && t < nc0 + c) {
      scores[c * a.score_stride + t] = v;
      if (a.hist) {
        const int dg = score_digit(v);
        atomicAdd(&hist[c * (NBINS / 2) + (dg >> 1)], 1u << ((dg & 1) << 4));
      }
    }
  };
#pragma unroll
  for (int i = 0; i < NS - 1; ++i)
    if (i < ntiles) issue(i);
  for (int i = 0; i < ntiles; ++i) {
    wait_ring<LPM>(min(NS - 2, ntiles - 1 - i));
    if (NWV > 1) __syncthreads();
    if (i + NS - 1 < ntiles) issue(i + NS - 1);
    const unsigned char* stg = smem + (i % NS) * SB;
    const int t0 = t_begin + (ntiles - 1 - i) * TW;
    t0_tile = t0;
    unsigned char* tile_k = smem + NS * SB;
    if constexpr (PS::KCONV) {
      convert_rows_e4m3<TW, 64 * NWV, HDIM>(stg, tile_k, tid);
      __syncthreads();  // the K tile converted by every wave
    }
    // logits S = Q.K^T of 16-token block bi for this wave's row tiles
    auto block_acc = [&](int bi, f32x4 (&acc)[RPW]) __attribute__((always_inline)) {
      const int row = 16 * bi + (lane & 15);
      uint4 k4[NKK];
      if constexpr (PS::KCONV) {
        const unsigned char* rp = tile_k + row * SRB;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
          k4[kk] = *(const uint4*)(rp + 16 * (k_chunk(kk, lane) ^ stage_swz(row)));
      } else if constexpr (KV8) {
#pragma unroll
        for (int i = 0; i < NKK / 2; ++i) k_operands_e4m3<RB>(stg, row, i, lane, k4[2 * i], k4[2 * i + 1]);
      } else {
        const unsigned char* rp = stg + row * SRB;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
          k4[kk] = *(const uint4*)(rp + 16 * (k_chunk(kk, lane) ^ stage_swz(row)));
      }
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) {
        acc[rr] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) acc[rr] = mfma_k32(q[rr][kk], k4[kk], acc[rr]);
      }
    };
    if constexpr (PS::PACK2) {
      // two blocks per emit: lane group j holds block bp + (j & 1); with 8
      // heads per query groups 0, 1 hold query 2 rt0 and groups 2, 3 query
      // 2 rt0 + 1, with 16 heads groups 2, 3 repeat groups 0, 1 (query rt0)
      const int q4 = lane >> 4;
#pragma unroll
      for (int bp = 0; bp < NB; bp += 2) {
        f32x4 acc_a[1], acc_b[1];
        block_acc(bp, acc_a);
        block_acc(bp + 1, acc_b);
        const float v = pool_pair_value<GP>(acc_a[0], acc_b[0], c2, fac[0], msub[0]);
        if (GP == 8 || q4 < 2) emit(v, GP == 8 ? 2 * rt0 + (q4 >> 1) : rt0, t0 + 16 * (bp + (q4 & 1)) + (lane & 15));
      }
    } else {
#pragma unroll
      for (int bi = 0; bi < NB; ++bi) {
        f32x4 acc[RPW];
        block_acc(bi, acc);
        if constexpr (PS::WPQ == 1)
          pool_emit_block<RPW, GP>(acc, c2, fac, msub, rt0, t0 + 16 * bi + (lane & 15), lane, emit);
        else
          pool_emit_block<RPW, GP>(acc, c2, fac, msub, rt0, t0 + 16 * bi + (lane & 15), lane, emit_part);
      }
    }
    if constexpr (PS::WPQ > 1) {  // the query's first wave adds its waves' parts and emits
      __syncthreads();
      if (wave % PS::WPQ == 0 && lane < TW) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < PS::WPQ; ++w) v += s_part[(wave + w) * TW + lane];
        emit(v, wave / PS::WPQ, t0 + lane);
      }
    }
  }
  __syncthreads();
  if (!a.hist) return;
  const int64_t row_c0 = ((int64_t)b * a.Hkv + g) * a.C;  // selection row of query 0
  for (int i = tid; i < a.C * (NBINS / 2); i += 64 * NWV) {
    const uint32_t v = hist[i];
    if (!v) continue;
    const int c = i / (NBINS / 2), w = i % (NBINS / 2);
    uint32_t* gh = a.hist + (row_c0 + c) * NBINS + 2 * w;
    if (v & 0xFFFFu) atomicAdd(gh, v & 0xFFFFu);
    if (v >> 16) atomicAdd(gh + 1, v >> 16);
  }
}

// Scores from the logits the full-attention ring kernel stored (small row
// counts: C * G logits per token cost less traffic than re-reading K):
// P = sum over h of exp2(s2_h - msub) * fac, the same constants as k_pool.
// grid (chunks of split_tokens tokens, B * Hkv; the host sizes the chunks,
// 1024-4096 tokens, for about two workgroups per CU), 256 threads, 4
// consecutive tokens per thread; dynamic LDS: C packed histograms.
__global__ __launch_bounds__(NT) void k_pool_logits(PoolArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint32_t* hist = (uint32_t*)smem;  // [C][NBINS/2], 16-bit packed counters
  __shared__ float s_fac[16], s_msub[16];
  const int64_t unit = blockIdx.y;
  const int b = (int)(unit / a.Hkv), g = (int)(unit % a.Hkv);
  const int tid = threadIdx.x;
  const int Lv = clamp_len(a.len, b, a.max_len);
  const int n_cand_max = Lv - a.W;  // union of the queries' candidates
  const int t_begin = blockIdx.x * a.split_tokens;
  if (t_begin >= n_cand_max) return;
  const int t_end = min(n_cand_max, t_begin + a.split_tokens);
  const int CG = a.C * a.G;
  for (int i = tid; i < a.C * (NBINS / 2); i += NT) hist[i] = 0;
  if (tid < CG) {
    const int c = tid / a.G, h = tid % a.G;
    const int64_t orow = ((int64_t)b * a.C + c) * a.Hq + (int64_t)g * a.G + h;
    const float m2 = a.stats_log2[orow * 2], z = a.stats_log2[orow * 2 + 1];
    const bool big = !(fabsf(m2) < 64.f);
    s_fac[tid] = z > 0.f ? (big ? 1.f / z : fast_exp2(-m2) / z) : 0.f;
    s_msub[tid] = (z > 0.f && big) ? m2 : 0.f;
  }
  __syncthreads();
  const int nc0 = Lv - a.C - a.W + 1;  // candidates of query 0 (query c: nc0 + c)
  const float* lg = a.logits + unit * CG * a.logit_stride;
  for (int t = t_begin + 4 * tid; t < t_end; t += 4 * NT) {
    for (int c = 0; c < a.C; ++c) {
      const int nc = nc0 + c;
      if (t >= nc) continue;  // not a candidate of query c (later queries have more)
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
      for (int h = 0; h < a.G; ++h) {
        const int r = c * a.G + h;
        const float4 l = *(const float4*)(lg + r * a.logit_stride + t);
        const float f = s_fac[r], m = s_msub[r];
        acc.x += fast_exp2(l.x - m) * f;
        acc.y += fast_exp2(l.y - m) * f;
        acc.z += fast_exp2(l.z - m) * f;
        acc.w += fast_exp2(l.w - m) * f;
      }
      float* sr = a.scores + (unit * a.C + c) * a.score_stride + t;
      const float v[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (t + j < nc) {
          sr[j] = v[j];
          if (a.hist) {
            const int dg = score_digit(v[j]);
            atomicAdd(&hist[c * (NBINS / 2) + (dg >> 1)], 1u << ((dg & 1) << 4));
          }
        }
    }
  }
  __syncthreads();
  if (!a.hist) return;
  for (int i = tid; i < a.C * (NBINS / 2); i += NT) {
    const uint32_t v = hist[i];
    if (!v) continue;
    const int c = i / (NBINS / 2), w = i % (NBINS / 2);
    uint32_t* gh = a.hist + (unit * a.C + c) * NBINS + 2 * w;
    if (v & 0xFFFFu) atomicAdd(gh, v & 0xFFFFu);
    if (v >> 16) atomicAdd(gh + 1, v >> 16);
  }
}

// ============================================================================ selection
// Per selection row (b, g, c): N candidates [0, pos - W + 1), k_eff = min(k, N).
struct RowInfo {
  int pos, N, keff;
};
__device__ inline RowInfo row_info(const SelArgs& a, int64_t row) {
  const int r = (int)row;  // rows = B Hkv C fit an int (checked by the host)
  const int c = r % a.C;
  const int b = r / (a.C * a.Hkv);
  const int Lv = clamp_len(a.len, b, a.max_len);
  RowInfo ri;
  ri.pos = Lv - a.C + c;
  ri.N = ri.pos - a.W + 1;
  if (ri.N < 0) ri.N = 0;
  ri.keff = a.k < ri.N ? a.k : ri.N;
  return ri;
}

__global__ void k_sel_init(SelArgs a) {
  const int64_t nh = a.rows * NBINS, ns = a.rows * 8;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nh + ns; i += (int64_t)gridDim.x * blockDim.x) {
    if (i < nh) a.hist[i] = 0;
    else a.state[i - nh] = 0;
  }
}

// Histogram of caller-given scores (hs2_select_from_scores): grid (chunks, rows).
__global__ __launch_bounds__(NT) void k_sel_hist(SelArgs a) {
  __shared__ uint32_t h[NBINS];
  const int64_t row = blockIdx.y;
  const RowInfo ri = row_info(a, row);
  const int t0 = blockIdx.x * SEL_CHUNK;
  if (t0 >= ri.N) return;
  const int t1 = min(ri.N, t0 + SEL_CHUNK);
  for (int i = threadIdx.x; i < NBINS; i += NT) h[i] = 0;
  __syncthreads();
  const float* P = a.scores + row * a.score_stride;
  for (int t = t0 + threadIdx.x; t < t1; t += NT) atomicAdd(&h[score_digit(P[t])], 1u);
  __syncthreads();
  for (int i = threadIdx.x; i < NBINS; i += NT)
    if (h[i]) atomicAdd(&a.hist[row * NBINS + i], h[i]);
}

// Exclusive scan over a 1024-thread block; returns the prefix, sets total.
__device__ inline int block_scan_1024(int v, int* lds16, int& total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds16[w] = x;
  __syncthreads();
  if (w == 0) {
    int s = lane < 16 ? lds16[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int y = __shfl_up(s, o);
      if (lane >= o) s += y;
    }
    if (lane < 16) lds16[lane] = s;
  }
  __syncthreads();
  const int off = w ? lds16[w - 1] : 0;
  total = lds16[15];
  __syncthreads();
  return off + x - v;
}

// Selection from the pooled scores and their histogram, in two launches
// (every workgroup of a row derives the same threshold bin b* and
// need = k_eff - #(keys in bins above b*)):
//   k_sel_filter  grid (chunks of 8192 tokens, rows), 256 threads: marks the
//                 tokens above b* in the row bitmap (raw-bit compares, one
//                 ballot per 64-token word) and collects the tokens of b*
//                 (gathered in LDS, one global slot reservation per
//                 workgroup);
//   k_sel_finish  grid (rows), 1024 threads: selects the `need` largest
//                 candidates by (key desc, index asc), i.e. by the 64-bit
//                 composite (key << 32) | ~index, with an 11-bit radix
//                 select over the bits b* leaves open that stops at the
//                 first digit whose keys are all taken, sets their bits (in
//                 an LDS copy of the row's bitmap, rows up to 512K tokens),
//                 then emits the bitmap's tokens in ascending order, the
//                 window, and -1 padding.
// state: [3] candidates collected (starts at zero).
constexpr int SELB = 1024;              // threads per selection workgroup
constexpr int SEL_PER = 16;             // tokens per thread
constexpr int SEL_TOKENS = SELB * SEL_PER;
constexpr int SEL_LDS_CAND = 2048;      // candidates a one-row workgroup (k_sel_fused) gathers in LDS
constexpr int RESOLVE_LDS_CAP = 6144;   // candidates the resolver keeps in LDS
constexpr size_t SEL_BM_LDS_MAX = 65536; // largest row bitmap kept in LDS (524288 tokens)
// longest rows selected by one workgroup (one chunk: with two, the 32K
// decode's selection was 1.4 us slower than the two-kernel path)
constexpr int SEL_FUSED_TOKENS = SEL_PER * SELB;
static_assert(NBINS == SELB, "one histogram bin per thread");

constexpr int RDX_BITS = 11;             // digit width of the candidates' radix select
constexpr int RDX_BINS = 1 << RDX_BITS;  // two histogram bins per thread
static_assert(RDX_BINS == 2 * SELB, "two radix bins per thread");

// A workgroup's LDS list of threshold-bin tokens (n counts every claimed
// slot, also those past the capacity, which went to global slots).
template <int CAP>
struct CandList {
  uint32_t key[CAP];
  int32_t idx[CAP];
  int n;
};

struct SelShared {
  union {
    CandList<SEL_LDS_CAND> cand;
    uint64_t comp[RESOLVE_LDS_CAP];
  } u;
  uint32_t h[RDX_BINS];
  uint64_t small[64];  // the threshold's digit bucket, when it is this small
  uint64_t thresh;
  int lds16[16];
  int base, digit, rem, all, bucket, nsmall, th[2];
};

struct Threshold {
  int mode, bstar, need;  // mode 0: nothing to select, 1: every candidate, 2: threshold bin
};

// cnt: this thread's bin NBINS - 1 - threadIdx.x of the row's histogram
// (bins from the top), loaded by the caller.
__device__ inline Threshold find_threshold(int cnt, const RowInfo& ri, SelShared& sh) {
  Threshold th{0, -1, 0};
  if (ri.keff == 0) return th;
  if (ri.keff == ri.N) {
    th.mode = 1;
    return th;
  }
  const int tid = threadIdx.x;
  if (tid == 0) {  // defaults if the histogram held fewer than k_eff keys (it cannot)
    sh.th[0] = 0;
    sh.th[1] = 0;
  }
  int total;
  const int above = block_scan_1024(cnt, sh.lds16, total);
  if (above < ri.keff && above + cnt >= ri.keff) {
    sh.th[0] = NBINS - 1 - tid;
    sh.th[1] = ri.keff - above;
  }
  __syncthreads();
  th.mode = 2;
  th.bstar = sh.th[0];
  th.need = sh.th[1];
  return th;
}
__device__ inline Threshold find_threshold(const SelArgs& a, int64_t row, const RowInfo& ri, SelShared& sh) {
  return find_threshold((int)a.hist[row * NBINS + NBINS - 1 - threadIdx.x], ri, sh);
}

// The digit tests of a row on the raw score bits x (a signed integer), for
// mode 2 (threshold bin b*): score_digit(x) > b*  <=>  x > above_gt and
// score_digit(x) >= b*  <=>  x >= cand_ge.  score_digit floors x by
// 2^DIGIT_SHIFT and clamps the result to [DIGIT_BASE, DIGIT_BASE + NBINS - 1],
// so for 1 <= d <= NBINS - 1 the digit is at least d exactly when
// x >= (d + DIGIT_BASE) << DIGIT_SHIFT; every digit is at least 0 (cand_ge
// the smallest int) and none exceeds NBINS - 1 (above_gt the largest).
struct DigitBounds {
  int above_gt, cand_ge, mode;
};
__device__ inline DigitBounds digit_bounds(const Threshold& th) {
  DigitBounds d{0x7FFFFFFF, 0x7FFFFFFF, th.mode};
  if (th.mode == 2) {
    if (th.bstar < NBINS - 1) d.above_gt = ((th.bstar + 1 + DIGIT_BASE) << DIGIT_SHIFT) - 1;
    d.cand_ge = th.bstar > 0 ? (th.bstar + DIGIT_BASE) << DIGIT_SHIFT : (int)0x80000000;
  }
  return d;
}

// Where the radix select over a row's candidates starts.  With
// 1 <= b* <= NBINS - 2 every candidate is a normal float whose key is its
// bits, with the top 32 - DIGIT_SHIFT bits equal to b* + DIGIT_BASE: the
// composites (key << 32) | ~index agree above bit 32 + DIGIT_SHIFT.
struct RadixStart {
  uint64_t prefix, pmask;
  int hi;  // composite bits [0, hi) are still open
};
__device__ inline RadixStart radix_start(int bstar) {
  if (bstar >= 1 && bstar <= NBINS - 2)
    return {(uint64_t)(bstar + DIGIT_BASE) << (32 + DIGIT_SHIFT), ~0ull << (32 + DIGIT_SHIFT), 32 + DIGIT_SHIFT};
  return {0ull, 0ull, 64};
}

// The need largest of the m candidates get their bitmap bits (in the row's
// LDS copy sbm when given, else in the global bitmap).  Radix select on the
// open composite bits, RDX_BITS at a time from the top; it stops at the
// first digit whose candidates are all taken.
__device__ inline void resolve_row(const SelArgs& a, int64_t row, int need, int m, const RadixStart& rs,
                                   SelShared& sh, uint64_t* sbm, bool comp_ready = false) {
  const int tid = threadIdx.x;
  const uint32_t* ck = a.cand_key + row * a.cand_cap;
  const int32_t* ci = a.cand_idx + row * a.cand_cap;
  uint32_t* bm32 = (uint32_t*)(a.bitmap + row * a.bitmap_words);
  if (need <= 0 || m <= 0) return;
  const bool in_lds = m <= RESOLVE_LDS_CAP;
  auto composite = [&](int i) -> uint64_t {
    return in_lds ? sh.u.comp[i] : (((uint64_t)ck[i] << 32) | (uint32_t)(~ci[i]));
  };
  if (in_lds && !comp_ready)  // (comp_ready: the caller built them in LDS)
    for (int i = tid; i < m; i += SELB) sh.u.comp[i] = ((uint64_t)ck[i] << 32) | (uint32_t)(~ci[i]);
  uint64_t thresh = 0;  // composite of the need-th largest (0: take every candidate)
  if (need < m) {
    uint64_t prefix = rs.prefix, pmask = rs.pmask;
    int rem = need;
    if (tid == 0) sh.nsmall = 0;  // (ordered before its use by the pass's barriers)
    for (int hi = rs.hi; hi > 0;) {
      const int width = hi < RDX_BITS ? hi : RDX_BITS;
      const int shift = hi - width;
      const uint32_t dmask = (1u << width) - 1u;
      sh.h[2 * tid] = 0;
      sh.h[2 * tid + 1] = 0;
      __syncthreads();
      for (int i = tid; i < m; i += SELB) {
        const uint64_t cv = composite(i);
        if ((cv & pmask) == prefix) atomicAdd(&sh.h[(uint32_t)(cv >> shift) & dmask], 1u);
      }
      __syncthreads();
      // thread t holds digits RDX_BINS - 1 - 2t and RDX_BINS - 2 - 2t (from the top)
      const int d1 = RDX_BINS - 1 - 2 * tid;
      const int h1 = (int)sh.h[d1], h0 = (int)sh.h[d1 - 1];
      int total;
      const int excl = block_scan_1024(h1 + h0, sh.lds16, total);  // keys with a larger digit
      if (excl < rem && excl + h1 >= rem) {
        sh.digit = d1;
        sh.rem = rem - excl;
        sh.bucket = h1;
        sh.all = h1 == rem - excl;  // the whole digit is taken
      } else if (excl + h1 < rem && excl + h1 + h0 >= rem) {
        sh.digit = d1 - 1;
        sh.rem = rem - excl - h1;
        sh.bucket = h0;
        sh.all = h0 == rem - excl - h1;
      }
      __syncthreads();
      prefix |= (uint64_t)sh.digit << shift;
      pmask |= (uint64_t)dmask << shift;
      rem = sh.rem;
      const bool done = sh.all;
      const int bucket = sh.bucket;
      __syncthreads();
      // every candidate under the prefix is taken: prefix with zero low bits
      // is the threshold (all larger composites are taken too)
      if (done) break;
      hi = shift;
      if (bucket <= 64 && in_lds) {
        // a small bucket: its rem-th largest composite (the one with exactly
        // rem - 1 larger in the bucket; composites are distinct) is the
        // threshold, ranked by one wave instead of further passes
        for (int i = tid; i < m; i += SELB) {
          const uint64_t cv = sh.u.comp[i];
          if ((cv & pmask) == prefix) sh.small[atomicAdd(&sh.nsmall, 1)] = cv;
        }
        __syncthreads();
        if (tid < bucket) {
          const uint64_t c = sh.small[tid];
          int larger = 0;
          for (int j = 0; j < bucket; ++j) larger += sh.small[j] > c;
          if (larger == rem - 1) sh.thresh = c;
        }
        __syncthreads();
        prefix = sh.thresh;
        break;
      }
    }
    thresh = prefix;
  } else {
    __syncthreads();
  }
  for (int i = tid; i < m; i += SELB) {
    const uint64_t cv = composite(i);
    if (cv >= thresh) {
      const int t = in_lds ? (int)~(uint32_t)cv : ci[i];
      if (sbm)
        atomicOr((unsigned long long*)&sbm[t >> 6], 1ull << (t & 63));
      else
        atomicOr(&bm32[t >> 5], 1u << (t & 31));
    }
  }
}

// Ascending emission into the row's index slots, two bitmap words per thread
// and block scan, from the row's LDS copy of the bitmap when given; else the
// global words are read with agent-scope atomic loads: this workgroup has
// just set bits in them with device atomics (ordered before these loads by
// the block barrier).
__device__ inline void emit_row(const SelArgs& a, int64_t row, const RowInfo& ri, SelShared& sh,
                                const uint64_t* sbm) {
  int32_t* out = a.idx + row * a.S;
  uint64_t* bm = a.bitmap + row * a.bitmap_words;
  const int tid = threadIdx.x;
  const int nwords = (ri.N + 63) >> 6;
  auto word = [&](int w) -> uint64_t {
    if (w >= nwords) return 0ull;
    uint64_t bits = sbm ? sbm[w] : __hip_atomic_load(&bm[w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (w == nwords - 1 && (ri.N & 63)) bits &= (1ull << (ri.N & 63)) - 1ull;  // tail bits are not maintained
    return bits;
  };
  int base = 0;
  for (int w0 = 0; w0 < nwords; w0 += 2 * SELB) {
    const int w = w0 + 2 * tid;
    uint64_t b0 = word(w), b1 = word(w + 1);
    int total;
    int p = base + block_scan_1024(__popcll(b0) + __popcll(b1), sh.lds16, total);
    while (b0) {
      const int bit = __ffsll((long long)b0) - 1;
      b0 &= b0 - 1;
      if (p < a.S) out[p] = 64 * w + bit;
      ++p;
    }
    while (b1) {
      const int bit = __ffsll((long long)b1) - 1;
      b1 &= b1 - 1;
      if (p < a.S) out[p] = 64 * (w + 1) + bit;
      ++p;
    }
    base += total;
  }
  const int wlo = ri.pos - a.W + 1 < 0 ? 0 : ri.pos - a.W + 1;
  const int nw = ri.pos >= 0 ? ri.pos - wlo + 1 : 0;
  for (int j = tid; j < nw; j += SELB)
    if (base + j < a.S) out[base + j] = wlo + j;
  for (int j = base + nw + tid; j < a.S; j += SELB) out[j] = -1;
}

// Raw score bits of the wave's NW words from token wt0 (row scores P,
// tokens below t1 read): v[j] holds token wt0 + 64 j + lane.
template <int NW>
__device__ inline void load_wave(const float* P, int wt0, int t1, int (&v)[NW]) {
  const int lane = threadIdx.x & 63;
  const int* src = (const int*)P + wt0;
  const int n = t1 - wt0;  // tokens from src on that may be read
  if (n >= 64 * NW) {
#pragma unroll
    for (int j = 0; j < NW; ++j) v[j] = src[64 * j + lane];
  } else {
#pragma unroll
    for (int j = 0; j < NW; ++j) v[j] = 64 * j + lane < n ? src[64 * j + lane] : 0;
  }
}

// Filters one wave's NW bitmap words from token wt0 (v from load_wave).  A
// word's taken bits are one compare's ballot and its threshold-bin tokens
// another's; both masks are parked in lane j of two register pairs, the
// taken words stored by lanes 0 .. NW - 1 together
// (bm: global or LDS).  The threshold-bin tokens then get consecutive slots:
// in the workgroup's LDS list cl when CAP > 0 (past its capacity, and always
// when CAP == 0, in global slots reserved in state[3]).  FAST: mode 2 and
// every token of the NW words valid (no validity masks).
template <bool FAST, int CAP, int NW>
__device__ inline void filter_wave(const SelArgs& a, int64_t row, const DigitBounds& db, int wt0, int t1,
                                   const int (&v)[NW], CandList<CAP>* cl, int* st, uint64_t* bm) {
  static_assert(NW <= 64, "one word per lane");
  const int lane = threadIdx.x & 63;
  int wlo = 0, whi = 0, clo = 0, chi = 0;
  int count = 0;  // threshold-bin tokens of the wave
#pragma unroll
  for (int j = 0; j < NW; ++j) {
    uint64_t sm, cm;
    if constexpr (FAST) {
      sm = __ballot(v[j] > db.above_gt);
      cm = __ballot(v[j] >= db.cand_ge) & ~sm;
    } else {
      const int tb = wt0 + 64 * j;
      if (tb >= t1) break;  // uniform across the wave
      const uint64_t vm = t1 - tb >= 64 ? ~0ull : (1ull << (t1 - tb)) - 1ull;
      sm = db.mode == 1 ? vm : (db.mode == 2 ? __ballot(v[j] > db.above_gt) & vm : 0ull);
      cm = db.mode == 2 ? __ballot(v[j] >= db.cand_ge) & vm & ~sm : 0ull;
    }
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(wlo) : "s"((uint32_t)sm), "i"(j));
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(whi) : "s"((uint32_t)(sm >> 32)), "i"(j));
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(clo) : "s"((uint32_t)cm), "i"(j));
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(chi) : "s"((uint32_t)(cm >> 32)), "i"(j));
    count += __popcll(cm);
  }
  const int nw = FAST ? NW : min(NW, max(0, (t1 - wt0 + 63) >> 6));
  if (lane < nw) bm[(wt0 >> 6) + lane] = ((uint64_t)(uint32_t)whi << 32) | (uint32_t)wlo;
  if (count == 0) return;  // uniform
  // slots [off, off + count): below CAP in LDS, the rest in global slots
  // reserved here from gbase on
  int off = 0, gbase = 0;
  if constexpr (CAP > 0) {
    if (lane == 0) off = atomicAdd(&cl->n, count);
    off = __builtin_amdgcn_readfirstlane(off);
  }
  const int excess = off + count - max(off, CAP);
  if (excess > 0) {
    if (lane == 0) gbase = atomicAdd(&st[3], excess);
    gbase = __builtin_amdgcn_readfirstlane(gbase);
  }
  uint32_t* ck = a.cand_key + row * a.cand_cap;
  int32_t* ci = a.cand_idx + row * a.cand_cap;
  int run = off;
#pragma unroll
  for (int j = 0; j < NW; ++j) {
    const uint64_t cm = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(chi, j) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane(clo, j);
    if (cm) {  // uniform
      if ((cm >> lane) & 1ull) {
        const int slot = run + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(cm >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)cm, 0u));
        const uint32_t key = score_key(__int_as_float(v[j]));
        const int t = wt0 + 64 * j + lane;
        if (CAP > 0 && slot < CAP) {
          cl->key[slot] = key;
          cl->idx[slot] = t;
        } else {
          const int gs = gbase + slot - max(off, CAP);
          ck[gs] = key;
          ci[gs] = t;
        }
      }
      run += __popcll(cm);
    }
  }
}

// The threshold of a row by one wave (the filter's workgroups are small):
// lane l holds bins NBINS - 16 - 16 l .. NBINS - 1 - 16 l (load_hist16, issued
// with the score loads); a wave scan gives the keys above each lane's bins,
// and the lane whose bins reach k_eff walks them from the top.  Same result
// as find_threshold.
__device__ inline void load_hist16(const SelArgs& a, int64_t row, uint32_t (&c)[16]) {
  const int lane = threadIdx.x & 63;
  const uint4* h4 = (const uint4*)(a.hist + row * NBINS + NBINS - 16 - 16 * lane);  // ascending
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint4 x = h4[q];
    c[4 * q] = x.x;
    c[4 * q + 1] = x.y;
    c[4 * q + 2] = x.z;
    c[4 * q + 3] = x.w;
  }
}
__device__ inline void threshold_by_wave(const uint32_t (&c)[16], int keff, int* th2) {
  const int lane = threadIdx.x & 63;
  int sum = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) sum += (int)c[i];
  int incl = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  int above = incl - sum;
  if (lane == 0) {  // defaults if the histogram held fewer than k_eff keys (it cannot)
    th2[0] = 0;
    th2[1] = 0;
  }
  if (above < keff && incl >= keff) {  // one lane: the crossing is in its bins
#pragma unroll
    for (int i = 15; i >= 0; --i) {
      if (above + (int)c[i] >= keff) {
        th2[0] = NBINS - 16 - 16 * lane + i;
        th2[1] = keff - above;
        break;
      }
      above += (int)c[i];
    }
  }
}

constexpr int SELF = 256;                          // threads per filter workgroup
constexpr int SELF_WORDS = 32;                     // bitmap words per filter wave
constexpr int SELF_TOKENS = SELF * SELF_WORDS;     // tokens per filter workgroup
constexpr int SELF_LDS_CAND = 2048;                // candidates a filter workgroup gathers in LDS

// grid (chunks of SELF_TOKENS tokens, rows), SELF threads: small workgroups
// (up to eight per CU) whose score, histogram and length loads all leave
// before the first wait (the scores up to the row's max_len, which the row
// always holds); the threshold-bin tokens are gathered in LDS and leave in
// one coalesced copy per workgroup (scattered one-lane global stores cost
// as much as the rest of the filter where the bin is dense).
__global__ __launch_bounds__(SELF) void k_sel_filter(SelArgs a) {
  __shared__ CandList<SELF_LDS_CAND> cl;
  __shared__ int th2[2], base;
  const int64_t row = blockIdx.y;
  const int t0 = blockIdx.x * SELF_TOKENS;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wt0 = t0 + 64 * SELF_WORDS * wave;
  int v[SELF_WORDS];
  load_wave(a.scores + row * a.score_stride, wt0, a.max_len, v);
  uint32_t c[16];
  if (wave == 0) load_hist16(a, row, c);
  const RowInfo ri = row_info(a, row);
  if (t0 >= ri.N) return;  // uniform across the workgroup
  const int t1 = min(ri.N, t0 + SELF_TOKENS);
  const int tid = threadIdx.x;
  if (tid == 0) cl.n = 0;
  Threshold th{ri.keff == ri.N ? 1 : 0, -1, 0};
  if (ri.keff > 0 && ri.keff < ri.N && wave == 0) threshold_by_wave(c, ri.keff, th2);
  __syncthreads();  // the list initialised, th2 written
  if (ri.keff > 0 && ri.keff < ri.N) th = Threshold{2, th2[0], th2[1]};
  int* st = a.state + row * 8;
  if (wt0 < t1) {  // uniform across the wave
    const DigitBounds db = digit_bounds(th);
    uint64_t* bm = a.bitmap + row * a.bitmap_words;
    if (db.mode == 2 && wt0 + 64 * SELF_WORDS <= t1)
      filter_wave<true>(a, row, db, wt0, t1, v, &cl, st, bm);
    else
      filter_wave<false>(a, row, db, wt0, t1, v, &cl, st, bm);
  }
  __syncthreads();
  const int n = min(cl.n, SELF_LDS_CAND);
  if (n > 0) {
    if (tid == 0) base = atomicAdd(&st[3], n);
    __syncthreads();
    const int64_t dst = row * a.cand_cap + base;
    for (int i = tid; i < n; i += SELF) {
      a.cand_key[dst + i] = cl.key[i];
      a.cand_idx[dst + i] = cl.idx[i];
    }
  }
}

// BM_LDS: the row's bitmap is copied into dynamic LDS at the start (its
// loads overlap the histogram's) and completed and emitted there; otherwise
// (rows of more than 512K tokens) the global bitmap is used throughout.
template <bool BM_LDS>
__global__ __launch_bounds__(SELB) void k_sel_finish(SelArgs a) {
  __shared__ SelShared sh;
  extern __shared__ __align__(16) uint64_t sbm[];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x;
  // every independent load first: count, histogram bin, bitmap, length
  const int m = min(a.state[row * 8 + 3], (int)a.cand_cap);
  const int cnt = (int)a.hist[row * NBINS + NBINS - 1 - tid];
  const RowInfo ri = row_info(a, row);
  if constexpr (BM_LDS) {
    const uint64_t* bm = a.bitmap + row * a.bitmap_words;
    const int nwords = (ri.N + 63) >> 6;
    for (int w = tid; w < nwords; w += SELB) sbm[w] = bm[w];
  }
  // the candidates' composites (when they fit in LDS), loaded before the
  // threshold's scan so that the loads overlap its barriers
  constexpr int CR = RESOLVE_LDS_CAP / SELB;
  static_assert(CR * SELB == RESOLVE_LDS_CAP, "whole rounds of candidates");
  const bool comp_lds = m <= RESOLVE_LDS_CAP;
  uint64_t cv[CR];
  if (comp_lds) {
    const uint32_t* ck = a.cand_key + row * a.cand_cap;
    const int32_t* ci = a.cand_idx + row * a.cand_cap;
#pragma unroll
    for (int r = 0; r < CR; ++r) {
      const int i = tid + SELB * r;
      cv[r] = i < m ? ((uint64_t)ck[i] << 32) | (uint32_t)(~ci[i]) : 0ull;
    }
  }
  const Threshold th = find_threshold(cnt, ri, sh);
  if (comp_lds) {
#pragma unroll
    for (int r = 0; r < CR; ++r)
      if (tid + SELB * r < m) sh.u.comp[tid + SELB * r] = cv[r];
  }
  __syncthreads();  // LDS bitmap and composites complete (find_threshold may return before its barriers)
  if (th.mode == 2) resolve_row(a, row, th.need, m, radix_start(th.bstar), sh, BM_LDS ? sbm : nullptr, comp_lds);
  __syncthreads();
  emit_row(a, row, ri, sh, BM_LDS ? sbm : nullptr);
}

// Rows of at most SEL_FUSED_TOKENS candidates: one workgroup per row filters
// every chunk into an LDS bitmap and LDS candidate list, then selects and
// emits (one launch; the two-kernel path above serves longer rows, whose
// chunks need more workgroups).
__global__ __launch_bounds__(SELB) void k_sel_fused(SelArgs a) {
  __shared__ SelShared sh;
  extern __shared__ __align__(16) uint64_t sbm[];
  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(a, row);
  const float* P = a.scores + row * a.score_stride;
  int* st = a.state + row * 8;
  const int tid = threadIdx.x;
  if (tid == 0) sh.u.cand.n = 0;
  const Threshold th = find_threshold(a, row, ri, sh);
  const DigitBounds db = digit_bounds(th);
  __syncthreads();  // the list initialised (find_threshold may return before its barriers)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int t0 = 0; t0 < ri.N; t0 += SEL_TOKENS) {
    const int t1 = min(ri.N, t0 + SEL_TOKENS);
    const int wt0 = t0 + 64 * SEL_PER * wave;
    if (wt0 < t1) {  // uniform across the wave
      int v[SEL_PER];
      load_wave(P, wt0, t1, v);
      filter_wave<false, SEL_LDS_CAND>(a, row, db, wt0, t1, v, &sh.u.cand, st, sbm);
    }
  }
  __syncthreads();
  const int n = sh.u.cand.n;
  if (th.mode == 2 && n > 0) {
    if (n <= SEL_LDS_CAND) {  // every candidate in LDS: composites in place, through registers
      uint64_t cv[SEL_LDS_CAND / SELB];
#pragma unroll
      for (int r = 0; r < SEL_LDS_CAND / SELB; ++r) {
        const int i = tid + SELB * r;
        cv[r] = i < n ? ((uint64_t)sh.u.cand.key[i] << 32) | (uint32_t)(~sh.u.cand.idx[i]) : 0ull;
      }
      __syncthreads();
#pragma unroll
      for (int r = 0; r < SEL_LDS_CAND / SELB; ++r)
        if (tid + SELB * r < n) sh.u.comp[tid + SELB * r] = cv[r];
      __syncthreads();
      resolve_row(a, row, th.need, n, radix_start(th.bstar), sh, sbm, true);
    } else {  // the LDS part joins the overflow in global memory
      if (tid == 0) sh.base = atomicAdd(&st[3], SEL_LDS_CAND);
      __syncthreads();
      const int64_t dst = row * a.cand_cap + sh.base;
      for (int i = tid; i < SEL_LDS_CAND; i += SELB) {
        a.cand_key[dst + i] = sh.u.cand.key[i];
        a.cand_idx[dst + i] = sh.u.cand.idx[i];
      }
      __threadfence_block();
      __syncthreads();
      resolve_row(a, row, th.need, min(n, (int)a.cand_cap), radix_start(th.bstar), sh, sbm);
    }
  }
  __syncthreads();
  emit_row(a, row, ri, sh, sbm);
}

// ---------------------------------------------------------------------------- block-level selection
// The candidates [0, N) of a selection row (b, g, c) are cut into blocks of
// `block` tokens (the last one cut short at N); a block's score is the fp32
// sum of its candidates' scores (scores below FLT_MIN count as zero; fixed
// summation order).  k_block_sums writes every block's score key; then one
// workgroup per row finds the k / block best blocks (score descending, lower
// block first among equal scores) by an 8-bit radix select on the keys held
// in LDS and emits them in ascending order as their tokens, then the window,
// then -1 padding.  Every selected block but the last one in ascending order
// is whole, so block r of the ascending list starts at output slot r * block.
constexpr int BSEL_MAX_BLOCKS = 16384;  // block keys per row in LDS (64 KB)
constexpr int BSUM_TOKENS = 8192;       // tokens per workgroup of k_block_sums

__device__ inline bool block_row(const BlockSelArgs& a, int64_t row, int& pos, int& N) {
  const int c = (int)(row % a.C);
  const int b = (int)(row / ((int64_t)a.C * a.Hkv));
  pos = clamp_len(a.len, b, a.max_len) - a.C + c;
  N = max(0, pos - a.W + 1);
  return pos >= 0;
}

// grid (ceil(max_len / BSUM_TOKENS), rows), 256 threads: each thread sums 4
// consecutive tokens, block / 4 lanes butterfly-sum one block (block is a
// power of two in [16, 256], so blocks never straddle lanes of two waves).
__global__ __launch_bounds__(256) void k_block_sums(BlockSelArgs a) {
  const int64_t row = blockIdx.y;
  int pos, N;
  if (!block_row(a, row, pos, N)) return;
  const int t0 = blockIdx.x * BSUM_TOKENS;
  if (t0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int B = a.block, gl = B / 4;  // lanes per block
  const float* P = a.scores + row * a.score_stride;
  uint32_t* keys = a.keys + row * a.key_stride;
  constexpr int U = BSUM_TOKENS / 1024;
  float v[U][4];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = t0 + 1024 * u + 4 * tid;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[u][i] = t + i < N ? P[t + i] : 0.f;
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = t0 + 1024 * u + 4 * tid;
    float x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = v[u][i] < 1.17549435e-38f ? 0.f : v[u][i];
    float sum = (x[0] + x[1]) + (x[2] + x[3]);
    for (int o = 1; o < gl; o <<= 1) sum += __shfl_xor(sum, o);
    if ((lane & (gl - 1)) == 0 && t < N) keys[t / B] = score_key(sum);
  }
}

// grid (rows), 1024 threads; dynamic LDS: 4 bytes per block of the longest row
__global__ __launch_bounds__(SELB) void k_block_select(BlockSelArgs a) {
  extern __shared__ uint32_t bkey[];  // [nb] score keys, then [kb] selected blocks ascending
  __shared__ uint32_t hist[256];
  __shared__ int lds16[16];
  __shared__ int s_dig[2];
  const int64_t row = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  int pos, N;
  int32_t* out = a.idx + row * a.S;
  if (!block_row(a, row, pos, N)) {
    for (int i = tid; i < a.S; i += SELB) out[i] = -1;
    return;
  }
  const int B = a.block;  // power of two
  const int nb = (N + B - 1) / B;
  const int kb = min(a.k / B, nb);

  // 1. the row's block keys
  const uint32_t* keys = a.keys + row * a.key_stride;
  for (int j = tid; j < nb; j += SELB) bkey[j] = keys[j];
  __syncthreads();

  // 2. threshold key T: fewer than kb keys above it, at least kb at or above
  uint32_t prefix = 0, mask = 0;
  int need = kb;  // blocks still to take among those matching the prefix
  if (kb > 0 && kb < nb) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0;
      __syncthreads();
      for (int j = tid; j < nb; j += SELB) {
        const uint32_t key = bkey[j];
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wave == 0) {  // lane l holds digits 255 - 4 l .. 252 - 4 l (from the top)
        int cnt[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cnt[i] = (int)hist[255 - 4 * lane - i];
          sum += cnt[i];
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o);
          if (lane >= o) incl += y;
        }
        int above = incl - sum;
        if (above < need && incl >= need) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if (above + cnt[i] >= need) {
              s_dig[0] = 255 - 4 * lane - i;
              s_dig[1] = need - above;
              break;
            }
            above += cnt[i];
          }
        }
      }
      __syncthreads();
      prefix |= (uint32_t)s_dig[0] << shift;
      mask |= 255u << shift;
      need = s_dig[1];
      __syncthreads();
    }
  }
  const uint32_t T = prefix;  // with kb == nb every block is taken (need stays nb)

  // 3. selection flags of this thread's contiguous blocks, ranks, emission
  const int per = (nb + SELB - 1) / SELB;
  const int j0 = tid * per, j1 = min(nb, j0 + per);
  uint32_t sel = 0;
  if (kb > 0) {
    int eq = 0;
    if (kb < nb)
      for (int j = j0; j < j1; ++j) eq += bkey[j] == T;
    int total;
    int eq_before = block_scan_1024(eq, lds16, total);
    for (int j = j0; j < j1; ++j) {
      const uint32_t key = bkey[j];
      bool take = kb == nb || key > T;
      if (kb < nb && key == T) take = eq_before++ < need;
      if (take) sel |= 1u << (j - j0);
    }
  }
  int before_total;
  const int sel_before = block_scan_1024(__popc(sel), lds16, before_total);  // barriers: keys read
  uint32_t* list = bkey;  // the keys are no longer needed
  {
    int r = sel_before;
    for (int j = j0; j < j1; ++j)
      if (sel >> (j - j0) & 1u) list[r++] = (uint32_t)j;
  }
  __syncthreads();
  const int blk_tokens = kb == 0 ? 0 : (kb - 1) * B + min(B, N - (int)list[kb - 1] * B);
  for (int e = tid; e < kb * B; e += SELB) {
    const int t = (int)list[e / B] * B + (e & (B - 1));
    if (t < N) out[e] = t;
  }
  const int wlo = max(0, pos - a.W + 1);
  const int nwin = pos - wlo + 1;
  for (int i = tid; i < a.S - blk_tokens; i += SELB) out[blk_tokens + i] = i < nwin ? wlo + i : -1;
}

// ============================================================================ sparse attention
// grid (n_split, units = B * Hkv * C), 64 * NWV threads, dynamic LDS = NS
// stages of TW gathered rows of K and V + the split's index slice.  Rows are
// the G heads of KV head g for query c (RT row tiles).  The split's index
// entries are staged in LDS first; each stage then gathers its rows straight
// into the ring (per-lane addresses), invalid entries (< 0 or >= len) read
// row 0 and are masked out of the softmax.
template <int RT, int NWV, int TW, int NS, bool KV8, int HDIM>
__global__ __launch_bounds__(64 * NWV) void k_sa_ring(SaArgs a) {
  constexpr int RPW = RT / NWV;
  constexpr int NB = TW / 16;
  constexpr int NKK = HDIM / 32;
  constexpr int SRB = 2 * HDIM;                 // bytes of a bf16 stage row
  constexpr int RB = KV8 ? HDIM : SRB;          // bytes of a staged cache row
  constexpr int RPL = 1024 / RB;                // rows per 1 KB load
  constexpr int CPR = RB / 16;                  // 16-byte chunks per staged row
  constexpr int LPM = TW * RB / 1024 / NWV;
  constexpr int SB = 2 * TW * RB;
  static_assert(LPM >= 1 && TW * RB == 1024 * LPM * NWV, "whole 1 KB loads per wave and stage");
  extern __shared__ __align__(16) unsigned char smem[];
  int32_t* sidx = (int32_t*)(smem + NS * SB);  // [split_slots]

  const int split = blockIdx.x;
  const int64_t unit = blockIdx.y;
  const int c = (int)(unit % a.C);
  const int g = (int)((unit / a.C) % a.Hkv);
  const int b = (int)(unit / ((int64_t)a.C * a.Hkv));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Lv = clamp_len(a.len, b, a.max_len);
  const int s_begin = split * a.split_slots;
  const int s_end = min(a.n_slots, s_begin + a.split_slots);
  const int nslots = s_end - s_begin;
  const int ntiles = (nslots + TW - 1) / TW;
  const int rt0 = wave * RPW;

  const int32_t* irow = a.idx + unit * a.idx_stride + s_begin;
  for (int i = threadIdx.x; i < ntiles * TW; i += 64 * NWV) {
    int t = i < nslots ? irow[i] : -1;
    sidx[i] = (t >= 0 && t < Lv) ? t : -1;
  }
  uint4 q[RPW][NKK];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    const int h = 16 * (rt0 + rr) + (lane & 15);
    if (h < a.G) {
      const uint16_t* p = a.q + (((int64_t)b * a.C + c) * a.Hq + g * a.G + h) * HDIM;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) q[rr][kk] = *(const uint4*)(p + q_koff(kk, lane));
    } else {
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) q[rr][kk] = make_uint4(0, 0, 0, 0);
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_enc(0));
  __syncthreads();

  constexpr int ESZ = KV8 ? 1 : 2;  // bytes per cache element
  const int64_t kvoff = ((int64_t)b * a.stride_b + (int64_t)g * a.stride_h) * ESZ;
  const unsigned char* Kbg = (const unsigned char*)a.K + kvoff;
  const unsigned char* Vbg = (const unsigned char*)a.V + kvoff;
  const int64_t stride_t = a.stride_t * ESZ;
  const float c2 = KV8 ? a.c2 * a.k_scale[g] : a.c2;
  const uint32_t ring = lds_addr(smem);
  uint32_t vmask[NS];  // row-validity bits of each ring stage (wave-uniform)

  auto issue = [&](int tile) {
    const uint32_t base = ring + (uint32_t)((tile % NS) * SB);
    uint32_t mask = 0;
#pragma unroll
    for (int u = 0; u < LPM; ++u) {
      const int n = wave * LPM + u;
      const int row = RPL * n + lane / CPR;
      const int t = sidx[tile * TW + row];
      const int64_t off = (int64_t)(t < 0 ? 0 : t) * stride_t +
                          (KV8 ? 16 * ((lane % CPR) ^ raw_swz<RB>(row)) : 16 * ((lane % CPR) ^ stage_swz(row)));
      dma16(Kbg + off, __builtin_amdgcn_readfirstlane(base + 1024 * n));
      dma16(Vbg + off, __builtin_amdgcn_readfirstlane(base + TW * RB + 1024 * n));
      const uint64_t bal = __ballot(t >= 0);  // lanes CPR j .. hold row RPL n + j
#pragma unroll
      for (int j = 0; j < RPL; ++j) mask |= (uint32_t)((bal >> (CPR * j)) & 1ull) << (RPL * n + j);
    }
    return mask;
  };

  WaveState<RPW, HDIM> st;
  st.init();
#pragma unroll
  for (int i = 0; i < NS - 1; ++i)
    if (i < ntiles) vmask[i] = issue(i);
  for (int i = 0; i < ntiles; ++i) {
    wait_ring<2 * LPM>(min(NS - 2, ntiles - 1 - i));
    if (NWV > 1) __syncthreads();
    uint32_t m_i = 0;
#pragma unroll
    for (int k = 0; k < NS; ++k)
      if (k == i % NS) m_i = vmask[k];
    if (i + NS - 1 < ntiles) {
      const uint32_t mnew = issue(i + NS - 1);
#pragma unroll
      for (int k = 0; k < NS; ++k)
        if (k == (i + NS - 1) % NS) vmask[k] = mnew;
    }
    const unsigned char* stg = smem + (i % NS) * SB;
    if (NWV > 1) {  // every wave's row bits
      __shared__ uint32_t s_mask[NWV];
      if (lane == 0) s_mask[wave] = m_i;
      __syncthreads();
      m_i = 0;
#pragma unroll
      for (int w = 0; w < NWV; ++w) m_i |= s_mask[w];
    }
    f32x4 S[NB][RPW];
#pragma unroll
    for (int bi = 0; bi < NB; ++bi) {
      if constexpr (KV8)
        qk_block_e4m3<RPW, RB>(stg, bi, q, S[bi], lane);
      else
        qk_block_swz<RPW>(stg, bi, q, S[bi], lane);
    }
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
        for (int ii = 0; ii < 4; ++ii) {
          const int row = 16 * bi + 4 * (lane >> 4) + ii;
          S[bi][rr][ii] = ((m_i >> row) & 1u) ? S[bi][rr][ii] * c2 : -INFINITY;
        }
    PFrags<NB, RPW> pf;
    online_softmax(st, S, pf, lane);
    if constexpr (KV8)  // E4M3: K and V operands read raw and converted in registers
      pv_tile_e4m3<RPW, NB, HDIM, RB>(st, pf, stg + TW * RB, lane);
    else
      pv_tile<RPW, NB, HDIM>(st, pf, stg + TW * SRB, lane);
  }
  const int64_t slot_base_row = (unit * a.n_split + split) * (16 * RT);
  store_partial<RPW>(st, a.part_o, a.part_ml, slot_base_row, rt0, lane);
}

// ============================================================================ streaming-read probe
// The device's practical streaming-read rate, the ceiling the streaming
// kernels are measured against.  grid: any number of 256-thread
// workgroups; the n16 16-byte words of src are cut into contiguous
// per-workgroup slices.  MODE 0: register loads (8 in flight per lane), 1:
// the same non-temporal, 2: 16-byte direct-to-LDS loads of 1 KB per wave as
// the streaming kernels issue them (up to 8 in flight per wave into an 8 KB
// ring, each piece read back from LDS once it has landed), 3: the same
// non-temporal; 4 and 5: gathers -- the buffer is R records of 512 (mode
// 4) or 256 (mode 5) bytes, R a power of two (checked by the host), read in
// a scattered order, logical record r at position (r * 0x9E3779B97F4A7C15)
// mod R (an odd multiplier: a permutation), each 1 KB direct-to-LDS wave
// load covering 2 or 4 records, as a sparse layer gathers a token's K and V
// rows from an interleaved bf16 or E4M3 cache.  Every mode folds each 32-bit word of src exactly once
// (xor); workgroup w stores the fold of its slice to sink[w] (keeps the
// loads live and lets a test check that every word was read once: the xor
// of sink[0, gridDim.x) is the xor of the whole buffer).  No atomics: the
// same-address atomics of a whole grid serialise for ~0.2 ms.
template <int MODE>
__global__ __launch_bounds__(256) void k_stream_probe(const uint4* __restrict__ src, int64_t n16, uint32_t* sink) {
  __shared__ __align__(16) unsigned char ring[4 * 8 * 1024];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = max(lo, min(n16, lo + per));
  uint32_t acc = 0;
  int64_t i = lo + tid;  // register-load part: words i, i + 256, ...
  if constexpr (MODE < 2) {
    constexpr int U = 8;
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4* s4 = (const u32x4*)src;
    for (; i + (U - 1) * 256 < hi; i += U * 256) {
      u32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if constexpr (MODE == 1)
          v[u] = __builtin_nontemporal_load(&s4[i + u * 256]);
        else
          v[u] = s4[i + u * 256];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
  } else if constexpr (MODE >= 4) {
    constexpr int RW = MODE == 4 ? 32 : 16;  // 16-byte words per record
    constexpr int RPP = 64 / RW;             // records per 1 KB piece
    const int64_t R = n16 / RW;
    const uint64_t rmask = (uint64_t)R - 1;
    auto perm = [&](int64_t r) { return (int64_t)(((uint64_t)r * 0x9E3779B97F4A7C15ull) & rmask); };
    const int64_t rper = (R + gridDim.x - 1) / gridDim.x;
    const int64_t rlo = (int64_t)blockIdx.x * rper;
    const int64_t rhi = max(rlo, min(R, rlo + rper));
    const unsigned char* wring = ring + wave * 8 * 1024;
    const uint32_t wring_a = lds_addr(wring);
    const int64_t npieces = (rhi - rlo) / RPP;
    auto fold = [&](int64_t n) {
      const uint4 v = *(const uint4*)(wring + 1024 * (n & 7) + 16 * lane);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    };
    int64_t n = 0;
    for (int64_t j = wave; j < npieces; j += 4, ++n) {
      const int64_t rec = perm(rlo + RPP * j + lane / RW);
      dma16_p<false>(src + RW * rec + lane % RW, __builtin_amdgcn_readfirstlane(wring_a + 1024u * (uint32_t)(n & 7)));
      __builtin_amdgcn_s_waitcnt(vmcnt_enc(7));  // at most 7 outstanding: piece n - 7 has landed
      if (n >= 7) {
        fold(n - 7);
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): read back before the next load reuses the slot
      }
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_enc(0));
    for (int64_t m = n > 7 ? n - 7 : 0; m < n; ++m) fold(m);
    // the slice's records after its whole pieces (fewer than RPP): register loads
    for (int64_t k = rlo + RPP * npieces + tid / RW; k < rhi && tid < RPP * RW; k += RPP) {
      const uint4 v = src[RW * perm(k) + tid % RW];
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    i = hi;  // no word tail: the records cover the buffer
  } else {
    // wave w loads 1 KB pieces j = w, w + 4, ... of the slice (64 words
    // each): its n-th piece into slot n % 8 of its ring
    const unsigned char* wring = ring + wave * 8 * 1024;
    const uint32_t wring_a = lds_addr(wring);
    const int64_t npieces = (hi - lo) / 64;
    auto fold = [&](int64_t n) {
      const uint4 v = *(const uint4*)(wring + 1024 * (n & 7) + 16 * lane);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    };
    int64_t n = 0;
    for (int64_t j = wave; j < npieces; j += 4, ++n) {
      dma16_p<MODE == 3>(src + lo + 64 * j + lane, __builtin_amdgcn_readfirstlane(wring_a + 1024u * (uint32_t)(n & 7)));
      __builtin_amdgcn_s_waitcnt(vmcnt_enc(7));  // at most 7 outstanding: piece n - 7 has landed
      if (n >= 7) {
        fold(n - 7);
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): read back before the next load reuses the slot
      }
    }
    __builtin_amdgcn_s_waitcnt(vmcnt_enc(0));
    for (int64_t m = n > 7 ? n - 7 : 0; m < n; ++m) fold(m);
    i = lo + 64 * npieces + tid;  // the slice's words after its whole pieces
  }
  for (; i < hi; i += 256) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  acc ^= __shfl_xor(acc, 1);
  acc ^= __shfl_xor(acc, 2);
  acc ^= __shfl_xor(acc, 4);
  acc ^= __shfl_xor(acc, 8);
  acc ^= __shfl_xor(acc, 16);
  acc ^= __shfl_xor(acc, 32);
  __shared__ uint32_t s_fold[4];
  if (lane == 0) s_fold[wave] = acc;
  __syncthreads();
  if (tid == 0) sink[blockIdx.x] = s_fold[0] ^ s_fold[1] ^ s_fold[2] ^ s_fold[3];
}

// ============================================================================ host launchers
#define HS2_LAUNCH(kernel, grid, block, shmem, stream, arg) \
  hipLaunchKernelGGL(kernel, grid, block, shmem, (hipStream_t)(stream), arg)

// Full attention kernel variants (the planner's defaults: head dim 128 with
// RT = 1 -> 2, RT = 2 -> 5, RT = 4 -> 7, RT = 8 -> 1 (E4M3: 7);
// head dim 256 with RT = 4, 8 -> 8, else 6):
//   1: workgroup kernel (64-row stages shared by 4 or 8 waves), head dim 128
//   0, 2, 3, 5, 7: ring kernels of head dim 128; 6, 8: head dim 256
// Columns: variant, RT, waves per token group, stage rows, stages, token
// groups, head dim.
#define HS2_RING_VARIANTS(X)                                                        \
  X(0, 1, 1, 16, 4, 1, 128) X(0, 2, 1, 16, 4, 1, 128) X(0, 4, 2, 16, 4, 1, 128)     \
  X(2, 1, 1, 32, 3, 1, 128) X(2, 2, 1, 32, 3, 1, 128) X(2, 4, 2, 32, 3, 1, 128)     \
  X(3, 1, 1, 16, 3, 1, 128) X(3, 2, 1, 16, 3, 1, 128) X(3, 4, 2, 16, 3, 1, 128)     \
  X(5, 1, 1, 32, 3, 1, 128) X(5, 2, 1, 16, 3, 2, 128) X(5, 4, 2, 16, 3, 2, 128)     \
  X(6, 1, 1, 16, 3, 1, 256) X(6, 2, 2, 16, 3, 1, 256) X(6, 4, 4, 16, 3, 1, 256)     \
  X(7, 2, 2, 32, 2, 2, 128) X(7, 4, 4, 32, 2, 2, 128) X(7, 8, 8, 64, 2, 1, 128)     \
  X(8, 4, 4, 32, 2, 1, 256) X(8, 8, 8, 32, 2, 1, 256)

// a ring shape serves a cache format only if every wave loads whole 1 KB
// pieces of each stage (the kernel asserts it; other shapes are never built)
constexpr bool fa_ring_ok(int nwv, int tw, bool kv8, int hd) { return tw * (kv8 ? hd : 2 * hd) / 1024 / nwv >= 1; }

int fa_variant_head_dim(int RT, int variant, bool kv8) {
  if (variant == 1) return !kv8 && (RT == 1 || RT == 2 || RT == 4 || RT == 8) ? 128 : 0;  // workgroup kernel
#define HS2_RING_HD(v, rt, nwv, tw, ns, tgw, hd) \
  if (variant == v && RT == rt) return fa_ring_ok(nwv, tw, kv8, hd) ? hd : 0;
  HS2_RING_VARIANTS(HS2_RING_HD)
#undef HS2_RING_HD
  return 0;
}

int fa_split_align(int RT, int variant) {
#define HS2_RING_ALIGN(v, rt, nwv, tw, ns, tgw, hd) \
  if (variant == v && RT == rt) return 64 * tgw;
  HS2_RING_VARIANTS(HS2_RING_ALIGN)
#undef HS2_RING_ALIGN
  return 64;
}

int fa_ring_token_groups(int RT, int variant) {
#define HS2_RING_TGW(v, rt, nwv, tw, ns, tgw, hd) \
  if (variant == v && RT == rt) return tgw;
  HS2_RING_VARIANTS(HS2_RING_TGW)
#undef HS2_RING_TGW
  return 1;
}

int fa_token_groups(int RT, int variant) {
  if (variant != 1) return 1;
  switch (RT) {
    case 1: return FaShape<1>::TGN;
    case 2: return FaShape<2>::TGN;
    case 4: return FaShape<4>::TGN;
    default: return FaShape<8>::TGN;
  }
}

// The runtime's figure, capped so that each resident workgroup's LDS plus
// 1 KB fits in the 160 KB of a compute unit: kernels whose LDS divides
// 160 KB exactly time as if one workgroup fewer were resident.
static hipError_t occupancy_capped(int* wgs, const void* fn, int threads, size_t lds) {
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(wgs, fn, threads, lds);
  if (e == hipSuccess && lds > 0) *wgs = std::min(*wgs, (int)((160 * 1024) / (lds + 1024)));
  return e;
}

constexpr size_t fa_ring_lds(int rt, int nwv, int tw, int ns, int tgw, bool kv8, int hd) {
  return (size_t)fa_ring_lds_bytes(rt, nwv, tw, ns, tgw, kv8, hd);
}

template <int RT, int NWV, int TW, int NS, int TGW, bool KV8, int HDIM>
hipError_t fa_ring_occupancy(int* wgs) {
  if constexpr (!fa_ring_ok(NWV, TW, KV8, HDIM)) {
    *wgs = 0;
    return hipSuccess;
  } else {  // the cache policy changes no resource
    return occupancy_capped(wgs, (const void*)k_fa_ring<RT, NWV, TW, NS, TGW, KV8, HDIM, FA_CACHE_DEFAULT>, 64 * NWV * TGW,
                            fa_ring_lds(RT, NWV, TW, NS, TGW, KV8, HDIM));
  }
}

template <int RT, int NWV, int TW, int NS, int TGW, bool KV8, int HDIM, int KP>
hipError_t fa_ring_launch(const FaArgs& a, dim3 grid, hipStream_t s) {
  if constexpr (!fa_ring_ok(NWV, TW, KV8, HDIM) || !fa_cache_policy_built(RT, KP)) {
    return hipErrorInvalidValue;
  } else {
    HS2_LAUNCH((k_fa_ring<RT, NWV, TW, NS, TGW, KV8, HDIM, KP>), grid, dim3(64 * NWV * TGW),
               fa_ring_lds(RT, NWV, TW, NS, TGW, KV8, HDIM), s, a);
    return hipGetLastError();
  }
}

template <int RT, int NWV, int TW, int NS, int TGW, int HDIM>
hipError_t fa_ring_dispatch(const FaArgs& a, dim3 grid, hipStream_t s) {
  const bool kv8 = a.k_scale != nullptr;
  switch (a.cache_policy) {
#define HS2_KP_CASE(kp)                                                                   \
  case kp:                                                                                \
    return kv8 ? fa_ring_launch<RT, NWV, TW, NS, TGW, true, HDIM, kp>(a, grid, s)         \
               : fa_ring_launch<RT, NWV, TW, NS, TGW, false, HDIM, kp>(a, grid, s);
    HS2_KP_CASE(FA_CACHE_DEFAULT)
    HS2_KP_CASE(FA_STREAM_V)
    HS2_KP_CASE(FA_STREAM_KV)
    HS2_KP_CASE(FA_STREAM_K_HEAD)
#undef HS2_KP_CASE
    default: return hipErrorInvalidValue;
  }
}

template <int RT, int NWV, int TW, int NS, int TGW, bool KV8, int HDIM, int KP>
hipError_t fa_ring_allow_lds_kp(int bytes) {
  if constexpr (!fa_ring_ok(NWV, TW, KV8, HDIM) || !fa_cache_policy_built(RT, KP)) {
    return hipSuccess;
  } else {
    return hipFuncSetAttribute((const void*)k_fa_ring<RT, NWV, TW, NS, TGW, KV8, HDIM, KP>,
                               hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  }
}

template <int RT, int NWV, int TW, int NS, int TGW, bool KV8, int HDIM>
hipError_t fa_ring_allow_lds(int bytes) {
  hipError_t e = fa_ring_allow_lds_kp<RT, NWV, TW, NS, TGW, KV8, HDIM, FA_CACHE_DEFAULT>(bytes);
  if (e == hipSuccess) e = fa_ring_allow_lds_kp<RT, NWV, TW, NS, TGW, KV8, HDIM, FA_STREAM_V>(bytes);
  if (e == hipSuccess) e = fa_ring_allow_lds_kp<RT, NWV, TW, NS, TGW, KV8, HDIM, FA_STREAM_KV>(bytes);
  if (e == hipSuccess) e = fa_ring_allow_lds_kp<RT, NWV, TW, NS, TGW, KV8, HDIM, FA_STREAM_K_HEAD>(bytes);
  return e;
}

hipError_t fa_wgs_per_cu(int RT, int variant, bool kv8, int* wgs) {
  *wgs = 0;
#define HS2_RING_OCC(v, rt, nwv, tw, ns, tgw, hd)                                                      \
  if (variant == v && RT == rt)                                                                       \
    return kv8 ? fa_ring_occupancy<rt, nwv, tw, ns, tgw, true, hd>(wgs)                               \
               : fa_ring_occupancy<rt, nwv, tw, ns, tgw, false, hd>(wgs);
  HS2_RING_VARIANTS(HS2_RING_OCC)
#undef HS2_RING_OCC
  if (kv8 || variant != 1) return hipSuccess;  // E4M3 only through the ring kernels
  const size_t sm = (size_t)FA_STAGES * STAGE_BYTES;
  switch (RT) {
    case 1: return occupancy_capped(wgs, (const void*)k_fa_split<1>, 64 * FaShape<1>::NW, sm);
    case 2: return occupancy_capped(wgs, (const void*)k_fa_split<2>, 64 * FaShape<2>::NW, sm);
    case 4: return occupancy_capped(wgs, (const void*)k_fa_split<4>, 64 * FaShape<4>::NW, sm);
    case 8: return occupancy_capped(wgs, (const void*)k_fa_split<8>, 64 * FaShape<8>::NW, sm);
    default: return hipSuccess;
  }
}

hipError_t launch_fa_split(const FaArgs& a, int RT, int variant, hipStream_t s) {
  dim3 grid(a.sp.n_items);
#define HS2_RING_LAUNCH(v, rt, nwv, tw, ns, tgw, hd) \
  if (variant == v && RT == rt) return fa_ring_dispatch<rt, nwv, tw, ns, tgw, hd>(a, grid, s);
  HS2_RING_VARIANTS(HS2_RING_LAUNCH)
#undef HS2_RING_LAUNCH
  if (a.k_scale || variant != 1) return hipErrorInvalidValue;  // E4M3 only through the ring kernels
  const size_t sm = (size_t)FA_STAGES * STAGE_BYTES;
  switch (RT) {
    case 1: HS2_LAUNCH(k_fa_split<1>, grid, dim3(64 * FaShape<1>::NW), sm, s, a); break;
    case 2: HS2_LAUNCH(k_fa_split<2>, grid, dim3(64 * FaShape<2>::NW), sm, s, a); break;
    case 4: HS2_LAUNCH(k_fa_split<4>, grid, dim3(64 * FaShape<4>::NW), sm, s, a); break;
    case 8: HS2_LAUNCH(k_fa_split<8>, grid, dim3(64 * FaShape<8>::NW), sm, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int RT, int GP, bool KV8, int HDIM>
size_t pool_smem_bytes(int C) {
  return (size_t)PoolShape<RT, GP, KV8, HDIM>::LDS + (size_t)C * (NBINS / 2) * sizeof(uint32_t);
}

// pool kernels for every (row tiles, padded group) pair the planner can produce:
// RT = pow2(ceil(C * GP / 16)) with C <= 16 and C * GP <= 128
#define HS2_POOL_CASES(X)                                     \
  X(1, 1) X(1, 2) X(1, 4) X(1, 8) X(1, 16)                    \
  X(2, 1) X(2, 2) X(2, 4) X(2, 8) X(2, 16) X(2, 32)           \
  X(4, 4) X(4, 8) X(4, 16) X(4, 32) X(4, 64)                  \
  X(8, 8) X(8, 16) X(8, 32) X(8, 64)

hipError_t launch_pool_logits(const PoolArgs& a, hipStream_t s) {
  const int64_t chunks = ((int64_t)a.max_len + a.split_tokens - 1) / a.split_tokens;
  HS2_LAUNCH(k_pool_logits, dim3((unsigned)chunks, (unsigned)(a.B * a.Hkv)), dim3(NT),
             (size_t)a.C * (NBINS / 2) * sizeof(uint32_t), s, a);
  return hipGetLastError();
}

template <int RT, int GP, bool KV8, int HDIM>
hipError_t pool_occupancy(int* wgs, int C) {
  return occupancy_capped(wgs, (const void*)k_pool<RT, GP, KV8, HDIM>, 64 * PoolShape<RT, GP, KV8, HDIM>::NWV,
                          pool_smem_bytes<RT, GP, KV8, HDIM>(C));
}

hipError_t pool_wgs_per_cu(int RT, int Gp, int C, bool kv8, int hd, int* wgs) {
  *wgs = 0;
#define HS2_POOL_OCC(rt, gp)                                                              \
  if (RT == rt && Gp == gp) {                                                             \
    if (hd == 256) return kv8 ? pool_occupancy<rt, gp, true, 256>(wgs, C)                 \
                              : pool_occupancy<rt, gp, false, 256>(wgs, C);               \
    return kv8 ? pool_occupancy<rt, gp, true, 128>(wgs, C) : pool_occupancy<rt, gp, false, 128>(wgs, C); \
  }
  HS2_POOL_CASES(HS2_POOL_OCC)
#undef HS2_POOL_OCC
  return hipSuccess;
}

template <int RT, int GP, bool KV8, int HDIM>
hipError_t launch_pool_one(const PoolArgs& a, dim3 grid, int hc, hipStream_t s) {
  HS2_LAUNCH((k_pool<RT, GP, KV8, HDIM>), grid, dim3(64 * PoolShape<RT, GP, KV8, HDIM>::NWV),
             (pool_smem_bytes<RT, GP, KV8, HDIM>(hc)), s, a);
  return hipGetLastError();
}

hipError_t launch_pool(const PoolArgs& a, int RT, hipStream_t s) {
  dim3 grid(a.n_split, a.Hkv, a.B);
  const int hc = a.hist ? a.C : 0;  // histograms in LDS
  const bool kv8 = a.k_scale != nullptr;
#define HS2_POOL_LAUNCH(rt, gp)                                                               \
  if (RT == rt && a.Gp == gp) {                                                               \
    if (a.hd == 256) return kv8 ? launch_pool_one<rt, gp, true, 256>(a, grid, hc, s)          \
                                : launch_pool_one<rt, gp, false, 256>(a, grid, hc, s);        \
    return kv8 ? launch_pool_one<rt, gp, true, 128>(a, grid, hc, s)                           \
               : launch_pool_one<rt, gp, false, 128>(a, grid, hc, s);                         \
  }
  HS2_POOL_CASES(HS2_POOL_LAUNCH)
#undef HS2_POOL_LAUNCH
  return hipErrorInvalidValue;
}

// sparse-attention ring kernels: (RT, waves) per head dim; 32-row stages x 2
constexpr int SAR_TW = 32, SAR_NS = 2;
#define HS2_SA_SHAPES(X) X(1, 1, 128) X(2, 1, 128) X(4, 2, 128) X(1, 1, 256) X(2, 2, 256) X(4, 4, 256)

hipError_t set_pool_smem_limits() {
  // dynamic LDS above 64 KB must be allowed explicitly
  const int big = 150 * 1024;  // leaves room for static LDS; no kernel asks for more
  hipError_t e = hipSuccess;
  auto allow = [&](const void* fn) {
    if (e == hipSuccess) e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, big);
  };
#define HS2_POOL_ATTR(rt, gp)                           \
  allow((const void*)k_pool<rt, gp, false, 128>);       \
  allow((const void*)k_pool<rt, gp, true, 128>);        \
  allow((const void*)k_pool<rt, gp, false, 256>);       \
  allow((const void*)k_pool<rt, gp, true, 256>);
  HS2_POOL_CASES(HS2_POOL_ATTR)
#undef HS2_POOL_ATTR
  allow((const void*)k_block_select);
  if (e == hipSuccess)  // its static LDS is large: only the bitmap's own limit
    e = hipFuncSetAttribute((const void*)k_sel_finish<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)SEL_BM_LDS_MAX);
  allow((const void*)k_fa_split<1>);
  allow((const void*)k_fa_split<2>);
  allow((const void*)k_fa_split<4>);
  allow((const void*)k_fa_split<8>);
#define HS2_RING_ATTR(v, rt, nwv, tw, ns, tgw, hd)                                          \
  if (e == hipSuccess) e = fa_ring_allow_lds<rt, nwv, tw, ns, tgw, false, hd>(big);         \
  if (e == hipSuccess) e = fa_ring_allow_lds<rt, nwv, tw, ns, tgw, true, hd>(big);
  HS2_RING_VARIANTS(HS2_RING_ATTR)
#undef HS2_RING_ATTR
#define HS2_SA_ATTR(rt, nwv, hd)                                          \
  allow((const void*)k_sa_ring<rt, nwv, SAR_TW, SAR_NS, false, hd>);     \
  allow((const void*)k_sa_ring<rt, nwv, SAR_TW, SAR_NS, true, hd>);
  HS2_SA_SHAPES(HS2_SA_ATTR)
#undef HS2_SA_ATTR
  return e;
}

hipError_t launch_combine(const CombineArgs& a, int rows_per_unit, int64_t units, hipStream_t s) {
  if (a.hd == 256)
    HS2_LAUNCH(k_combine<256>, dim3(rows_per_unit, (unsigned)units), dim3(256), 0, s, a);
  else
    HS2_LAUNCH(k_combine<128>, dim3(rows_per_unit, (unsigned)units), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sel_init(const SelArgs& a, hipStream_t s) {
  const int64_t n = a.rows * (NBINS + 8);
  const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
  HS2_LAUNCH(k_sel_init, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_sel_hist(const SelArgs& a, int nchunks, hipStream_t s) {
  HS2_LAUNCH(k_sel_hist, dim3(nchunks, (unsigned)a.rows), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_block_select(const BlockSelArgs& a, hipStream_t s) {
  const size_t nb_max = ((size_t)a.max_len + a.block - 1) / a.block;
  if (nb_max > (size_t)BSEL_MAX_BLOCKS || a.key_stride < (int64_t)nb_max || a.block < 16 || a.block > 256 ||
      (a.block & (a.block - 1)))
    return hipErrorInvalidValue;
  const unsigned chunks = (unsigned)(((int64_t)a.max_len + BSUM_TOKENS - 1) / BSUM_TOKENS);
  HS2_LAUNCH(k_block_sums, dim3(chunks, (unsigned)a.rows), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  HS2_LAUNCH(k_block_select, dim3((unsigned)a.rows), dim3(SELB), nb_max * sizeof(uint32_t), s, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelArgs& a, hipStream_t s) {
  if (a.max_len <= SEL_FUSED_TOKENS) {
    HS2_LAUNCH(k_sel_fused, dim3((unsigned)a.rows), dim3(SELB), (size_t)a.bitmap_words * sizeof(uint64_t), s, a);
    return hipGetLastError();
  }
  const int64_t chunks = ((int64_t)a.max_len + SELF_TOKENS - 1) / SELF_TOKENS;
  HS2_LAUNCH(k_sel_filter, dim3((unsigned)chunks, (unsigned)a.rows), dim3(SELF), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t bm_bytes = (size_t)a.bitmap_words * sizeof(uint64_t);
  if (bm_bytes <= SEL_BM_LDS_MAX)
    HS2_LAUNCH(k_sel_finish<true>, dim3((unsigned)a.rows), dim3(SELB), bm_bytes, s, a);
  else
    HS2_LAUNCH(k_sel_finish<false>, dim3((unsigned)a.rows), dim3(SELB), 0, s, a);
  return hipGetLastError();
}

size_t sa_smem_bytes(int split_slots, bool kv8, int hd) {
  return (size_t)SAR_NS * 2 * SAR_TW * (kv8 ? hd : 2 * hd) +
         sizeof(int32_t) * (size_t)((split_slots + SAR_TW - 1) / SAR_TW * SAR_TW);
}

hipError_t launch_sa_split(const SaArgs& a, int RT, hipStream_t s) {
  dim3 grid(a.n_split, (unsigned)((int64_t)a.B * a.Hkv * a.C));
  const bool kv8 = a.k_scale != nullptr;
  const size_t sm = sa_smem_bytes(a.split_slots, kv8, a.hd);
#define HS2_SA_LAUNCH(rt, nwv, hdim)                                                                 \
  if (RT == rt && a.hd == hdim) {                                                                    \
    if (kv8)                                                                                         \
      HS2_LAUNCH((k_sa_ring<rt, nwv, SAR_TW, SAR_NS, true, hdim>), grid, dim3(64 * nwv), sm, s, a);  \
    else                                                                                             \
      HS2_LAUNCH((k_sa_ring<rt, nwv, SAR_TW, SAR_NS, false, hdim>), grid, dim3(64 * nwv), sm, s, a); \
    return hipGetLastError();                                                                        \
  }
  HS2_SA_SHAPES(HS2_SA_LAUNCH)
#undef HS2_SA_LAUNCH
  return hipErrorInvalidValue;
}

hipError_t launch_stream_probe(const void* src, int64_t n16, int mode, uint32_t* sink, hipStream_t s) {
  // 16 workgroups per compute unit of 256 (more than stay resident: the
  // dispatcher keeps every CU busy to the end), one sink word each
  const dim3 grid(STREAM_PROBE_WORKGROUPS), block(256);
  const uint4* p = (const uint4*)src;
  switch (mode) {
    case 0: hipLaunchKernelGGL(k_stream_probe<0>, grid, block, 0, s, p, n16, sink); break;
    case 1: hipLaunchKernelGGL(k_stream_probe<1>, grid, block, 0, s, p, n16, sink); break;
    case 2: hipLaunchKernelGGL(k_stream_probe<2>, grid, block, 0, s, p, n16, sink); break;
    case 3: hipLaunchKernelGGL(k_stream_probe<3>, grid, block, 0, s, p, n16, sink); break;
    case 4: hipLaunchKernelGGL(k_stream_probe<4>, grid, block, 0, s, p, n16, sink); break;
    case 5: hipLaunchKernelGGL(k_stream_probe<5>, grid, block, 0, s, p, n16, sink); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hs2
