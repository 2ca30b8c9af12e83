// HIP kernels of the hybrid-block decode path (gfx950).
//
//   k_fa_split   full attention, split-KV flash decode: per (sequence, KV head,
//                token split) partial (m, l, O) of every query row of the group
//   k_combine    merge of the partials -> bf16 output and (M, Z) per query row
//   k_pool       re-reads K, recomputes the same logits, turns them into exact
//                probabilities with the merged (M, Z) and sums them over the
//                query heads of the KV head -> pooled score per candidate token;
//                builds the first-level radix histogram of the scores
//   k_sel_*      top-k outside the window (radix select on the score keys,
//                ties to the lower index) + window union + ascending emission
//   k_sa_split   sparse attention over gathered selected rows (same partial
//                format, merged by k_combine)
//
// Query rows of one (sequence, KV head) group are laid out query-major:
// row r = c * Gp + h with Gp = G rounded up to a power of two; rows with
// h >= G or c >= C are padding (zero queries, never written out).
#include "hs2_device.h"
#include "hs2_launch.h"

namespace hs2 {

// ============================================================================ helpers
__device__ inline int clamp_len(const int32_t* len, int b, int max_len) {
  int L = len[b];
  return L < 0 ? 0 : (L > max_len ? max_len : L);
}

// Load B operands (Q^T) of query row tile rt for this lane: row 16 rt + (lane & 15).
__device__ inline void load_q_tile(uint4 (&q)[4], const uint16_t* __restrict__ qbase, int rt, int lane, int Gp,
                                   int G, int C, int Hq, int g, int b) {
  const int r = 16 * rt + (lane & 15);
  const int c = r / Gp, h = r % Gp;
  if (c < C && h < G) {
    const uint16_t* p = qbase + (((int64_t)b * C + c) * Hq + g * G + h) * HD + 8 * (lane >> 4);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) q[kk] = *(const uint4*)(p + 32 * kk);
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) q[kk] = make_uint4(0, 0, 0, 0);
  }
}

// ============================================================================ full attention
// grid (n_split, Hkv, B), 256 threads.  Waves split the work of one LDS tile:
// RT <= 2: TG = 4 / RT token groups, each wave one row tile and BPW = RT blocks;
// RT >= 4: each wave RT / 4 row tiles and all four 16-row blocks.
template <int RT>
__global__ __launch_bounds__(NT) void k_fa_split(FaArgs a) {
  constexpr int TG = RT >= 4 ? 1 : 4 / RT;
  constexpr int RPW = RT >= 4 ? RT / 4 : 1;
  constexpr int BPW = 4 / TG;
  constexpr int WPT = 4 / TG;  // waves per token group
  __shared__ TileLds lds;

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Lv = clamp_len(a.len, b, a.max_len);
  const int t_begin = split * a.split_tokens;
  if (t_begin >= Lv) return;
  const int t_end = min(Lv, t_begin + a.split_tokens);
  const int tg = wave / WPT;
  const int rt0 = (wave % WPT) * RPW;

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
  const int cg = tid & 15;

  WaveState<RPW> st;
  st.init();
  int blk[BPW];
#pragma unroll
  for (int bi = 0; bi < BPW; ++bi) blk[bi] = tg * BPW + bi;

  TileRegs regs;
  {
    int tok[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t_begin + row_of(tid, u);
      tok[u] = t < t_end ? t : -1;
    }
    load_tile<true>(regs, Kbg, Vbg, a.stride_t, tok, cg);
  }
  for (int t0 = t_begin; t0 < t_end; t0 += TILE) {
    __syncthreads();
    store_tile<true>(lds, regs, tid);
    __syncthreads();
    if (t0 + TILE < t_end) {
      int tok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = t0 + TILE + row_of(tid, u);
        tok[u] = t < t_end ? t : -1;
      }
      load_tile<true>(regs, Kbg, Vbg, a.stride_t, tok, cg);
    }
    f32x4 S[BPW][RPW];
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) qk_block<RPW>(lds, blk[bi], q, S[bi], lane);
    const bool full = (t0 + TILE <= t_end) && (t0 + TILE - 1 <= min_pos);
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi)
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = S[bi][rr][i] * a.c2;
          if (!full) {
            const int t = t0 + 16 * blk[bi] + 4 * (lane >> 4) + i;
            if (t >= t_end || t > rpos[rr]) v = -INFINITY;
          }
          S[bi][rr][i] = v;
        }
    softmax_pv<RPW, BPW>(st, lds, blk, S, lane);
  }
  const int nslot = a.n_split * TG;
  const int64_t unit = (int64_t)b * a.Hkv + g;
  const int64_t slot_base_row = (unit * nslot + (int64_t)split * TG + tg) * (16 * RT);
  store_partial<RPW>(st, a.part_o, a.part_ml, slot_base_row, rt0, lane);
}

// ============================================================================ combine
// grid (rows_per_unit, units), 128 threads (one per head-dim element).
// FA: unit = (b, g), row r = c * Gp + h; slots valid = ceil(Lv / split) * TG.
// SA: unit = (b, g, c), row = h; all n_split * TG slots written.
__global__ __launch_bounds__(HD) void k_combine(CombineArgs a) {
  const int r = blockIdx.x;
  const int64_t unit = blockIdx.y;
  const int d = threadIdx.x;
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
  if (!a.sa_mode) {
    const int Lv = clamp_len(a.len, b, a.max_len);
    nvalid = ((Lv + a.split_tokens - 1) / a.split_tokens) * a.tg;
  }
  const int64_t base = unit * a.nslot * a.rows;
  float M = -INFINITY;
  for (int s = 0; s < nvalid; ++s) M = fmaxf(M, a.part_ml[(base + (int64_t)s * a.rows + r) * 2]);
  float Z = 0.f, acc = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < nvalid; ++s) {
      const int64_t pr = base + (int64_t)s * a.rows + r;
      const float m = a.part_ml[pr * 2];
      if (m == -INFINITY) continue;
      const float w = fast_exp2(m - M);
      Z += a.part_ml[pr * 2 + 1] * w;
      acc += a.part_o[pr * HD + d] * w;
    }
  }
  const float o = Z > 0.f ? acc / Z : 0.f;
  const int64_t orow = ((int64_t)b * a.C + c) * a.Hq + (int64_t)g * a.G + h;
  a.out[orow * HD + d] = (uint16_t)f32_to_bf16_bits(o);
  if (d == 0) {
    if (a.stats_log2) {
      a.stats_log2[orow * 2] = M;
      a.stats_log2[orow * 2 + 1] = Z;
    }
    if (a.stats_user) {
      a.stats_user[orow * 2] = M == -INFINITY ? M : M * 0.69314718055994531f;
      a.stats_user[orow * 2 + 1] = Z;
    }
  }
}

// ============================================================================ pooled scores
// grid (n_split, Hkv, B), 256 threads; wave w handles 16-row block w of every
// LDS tile, for all RT query row tiles (queries read from LDS).
template <int RT>
__global__ __launch_bounds__(NT) void k_pool(PoolArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  TileLds& lds = *(TileLds*)smem;  // only the K part (first member) is allocated and used
  uint16_t* qs = (uint16_t*)(smem + KTILE_BYTES);                                   // [16 RT][KPAD]
  uint32_t* hist = (uint32_t*)(smem + KTILE_BYTES + 16 * RT * KPAD * sizeof(uint16_t));  // [C][NBINS/2]

  const int split = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Lv = clamp_len(a.len, b, a.max_len);
  // candidates of query c: [0, Lv - C + c - W + 1); the union over c ends at Lv - W
  const int n_cand_max = Lv - a.W;
  const int t_begin = split * a.split_tokens;
  if (t_begin >= n_cand_max) return;
  const int t_end = min(n_cand_max, t_begin + a.split_tokens);

  for (int i = tid; i < a.C * (NBINS / 2); i += NT) hist[i] = 0;
  for (int i = tid; i < 16 * RT * 16; i += NT) {
    const int r = i >> 4, cgq = i & 15;
    const int c = r / a.Gp, h = r % a.Gp;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (c < a.C && h < a.G) v = *(const uint4*)(a.q + (((int64_t)b * a.C + c) * a.Hq + g * a.G + h) * HD + cgq * 8);
    *(uint4*)&qs[r * KPAD + cgq * 8] = v;
  }
  // per-lane (M, 1/Z-free) stats of rows 16 rt + (lane & 15)
  float m2[RT], zr[RT];
  int ncand[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int r = 16 * rt + (lane & 15);
    const int c = r / a.Gp, h = r % a.Gp;
    if (c < a.C && h < a.G) {
      const int64_t orow = ((int64_t)b * a.C + c) * a.Hq + (int64_t)g * a.G + h;
      m2[rt] = a.stats_log2[orow * 2];
      zr[rt] = a.stats_log2[orow * 2 + 1];
      ncand[rt] = Lv - a.C + c - a.W + 1;
    } else {
      m2[rt] = 0.f;
      zr[rt] = 0.f;  // marks a padding row: contributes nothing
      ncand[rt] = 0;
    }
  }
  const int64_t kvoff = (int64_t)b * a.stride_b + (int64_t)g * a.stride_h;
  const uint16_t* Kbg = a.K + kvoff;
  const int cg = tid & 15;
  TileRegs regs;
  {
    int tok[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t_begin + row_of(tid, u);
      tok[u] = t < t_end ? t : -1;
    }
    load_tile<false>(regs, Kbg, nullptr, a.stride_t, tok, cg);
  }
  const int64_t row_c0 = ((int64_t)b * a.Hkv + g) * a.C;  // selection row of query 0
  for (int t0 = t_begin; t0 < t_end; t0 += TILE) {
    __syncthreads();
    store_tile<false>(lds, regs, tid);
    __syncthreads();
    if (t0 + TILE < t_end) {
      int tok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = t0 + TILE + row_of(tid, u);
        tok[u] = t < t_end ? t : -1;
      }
      load_tile<false>(regs, Kbg, nullptr, a.stride_t, tok, cg);
    }
    // logits of block `wave` against every row tile
    const uint16_t* kp = &lds.k[(16 * wave + (lane & 15)) * KPAD + 8 * (lane >> 4)];
    uint4 ka[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) ka[kk] = *(const uint4*)(kp + 32 * kk);
    const int tbase = t0 + 16 * wave + 4 * (lane >> 4);
    float e[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const uint16_t* qp = &qs[(16 * rt + (lane & 15)) * KPAD + 8 * (lane >> 4)];
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) acc = mfma_k32(ka[kk], *(const uint4*)(qp + 32 * kk), acc);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float s2 = acc[i] * a.c2;
        e[rt][i] = (zr[rt] > 0.f && tbase + i < ncand[rt]) ? fast_exp2(s2 - m2[rt]) / zr[rt] : 0.f;
      }
    }
    // sum over the heads of each query, then record candidates
    if (a.Gp <= 16) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = e[rt][i];
          for (int s = 1; s < a.Gp; s <<= 1) v += __shfl_xor(v, s);
          e[rt][i] = v;
        }
        const int r = 16 * rt + (lane & 15);
        const int c = r / a.Gp;
        if ((r % a.Gp) == 0 && c < a.C) {
          const int nc = Lv - a.C + c - a.W + 1;
          float* dst = a.scores + (row_c0 + c) * a.score_stride;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = tbase + i;
            if (t < nc) {
              dst[t] = e[rt][i];
              const int dg = score_digit(score_key(e[rt][i]));
              atomicAdd(&hist[c * (NBINS / 2) + (dg >> 1)], 1u << ((dg & 1) << 4));
            }
          }
        }
      }
    } else {
      const int tiles_per_q = a.Gp / 16;
      for (int c = 0; c < a.C; ++c) {
        float v[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          if (rt / tiles_per_q == c)
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] += e[rt][i];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          for (int s = 1; s < 16; s <<= 1) v[i] += __shfl_xor(v[i], s);
        if ((lane & 15) == 0) {
          const int nc = Lv - a.C + c - a.W + 1;
          float* dst = a.scores + (row_c0 + c) * a.score_stride;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int t = tbase + i;
            if (t < nc) {
              dst[t] = v[i];
              const int dg = score_digit(score_key(v[i]));
              atomicAdd(&hist[c * (NBINS / 2) + (dg >> 1)], 1u << ((dg & 1) << 4));
            }
          }
        }
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < a.C * (NBINS / 2); i += NT) {
    const uint32_t v = hist[i];
    if (!v) continue;
    const int c = i / (NBINS / 2), w = i % (NBINS / 2);
    uint32_t* gh = a.hist + (row_c0 + c) * NBINS + 2 * w;
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
  const int c = (int)(row % a.C);
  const int b = (int)(row / ((int64_t)a.C * a.Hkv));
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
  const int t0 = blockIdx.x * a.chunk;
  if (t0 >= ri.N) return;
  const int t1 = min(ri.N, t0 + a.chunk);
  for (int i = threadIdx.x; i < NBINS; i += NT) h[i] = 0;
  __syncthreads();
  const float* P = a.scores + row * a.score_stride;
  for (int t = t0 + threadIdx.x; t < t1; t += NT) atomicAdd(&h[score_digit(score_key(P[t]))], 1u);
  __syncthreads();
  for (int i = threadIdx.x; i < NBINS; i += NT)
    if (h[i]) atomicAdd(&a.hist[row * NBINS + i], h[i]);
}

// Find the bin holding the k_eff-th largest key: grid (rows), 256 threads.
// state: [0] mode (0 none, 1 all candidates, 2 threshold), [1] bin b*,
//        [2] need = k_eff - #(keys in bins above b*), [3] candidate count.
__global__ __launch_bounds__(NT) void k_sel_threshold(SelArgs a) {
  __shared__ int part[NT];
  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(a, row);
  int* st = a.state + row * 8;
  const int tid = threadIdx.x;
  if (ri.keff == 0 || ri.keff == ri.N) {
    if (tid == 0) {
      st[0] = ri.keff == 0 ? 0 : 1;
      st[1] = -1;
      st[2] = 0;
    }
    return;
  }
  // thread tid owns bins [NBINS - 8 (tid + 1), NBINS - 8 tid), scanned from the top
  const uint32_t* hr = a.hist + row * NBINS;
  int cnt[8], s = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    cnt[j] = (int)hr[NBINS - 1 - 8 * tid - j];
    s += cnt[j];
  }
  part[tid] = s;
  __syncthreads();
  if (tid == 0) {
    int acc = 0;
    for (int i = 0; i < NT; ++i) {
      const int v = part[i];
      part[i] = acc;  // exclusive prefix from the top
      acc += v;
    }
  }
  __syncthreads();
  int above = part[tid];
  if (above < ri.keff && above + s >= ri.keff) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (above + cnt[j] >= ri.keff) {
        st[0] = 2;
        st[1] = NBINS - 1 - 8 * tid - j;
        st[2] = ri.keff - above;
        break;
      }
      above += cnt[j];
    }
  }
}

// Mark tokens above the threshold bin in the row bitmap and collect the
// tokens of the threshold bin: grid (chunks, rows), 256 threads.
__global__ __launch_bounds__(NT) void k_sel_filter(SelArgs a) {
  const int64_t row = blockIdx.y;
  const RowInfo ri = row_info(a, row);
  const int t0 = blockIdx.x * a.chunk;
  if (t0 >= ri.N) return;
  const int t1 = min(ri.N, t0 + a.chunk);
  int* st = a.state + row * 8;
  const int mode = st[0], bstar = st[1];
  const float* P = a.scores + row * a.score_stride;
  uint64_t* bm = a.bitmap + row * a.bitmap_words;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int tb = t0 + 64 * wave; tb < t1; tb += 64 * (NT / 64)) {
    const int t = tb + lane;
    const bool valid = t < t1;
    bool sel = false, cand = false;
    uint32_t key = 0;
    if (valid && mode != 0) {
      key = score_key(P[t]);
      if (mode == 1) {
        sel = true;
      } else {
        const int d = score_digit(key);
        sel = d > bstar;
        cand = d == bstar;
      }
    }
    const uint64_t sm = __ballot(sel);
    if (lane == 0) bm[tb >> 6] = sm;
    const uint64_t cm = __ballot(cand);
    if (cm) {
      int basev = 0;
      if (lane == 0) basev = atomicAdd(&st[3], __popcll(cm));
      basev = __shfl(basev, 0);
      if (cand) {
        const int slot = basev + __popcll(cm & ((1ull << lane) - 1ull));
        a.cand_key[row * a.cand_cap + slot] = key;
        a.cand_idx[row * a.cand_cap + slot] = t;
      }
    }
  }
}

// Exact selection inside the threshold bin: the `need` largest of the
// candidates by (key desc, index asc), by radix select on the 64-bit
// composite key (key << 32) | ~index.  grid (rows), 1024 threads.
__global__ __launch_bounds__(1024) void k_sel_resolve(SelArgs a) {
  __shared__ uint32_t h[256];
  __shared__ uint64_t s_prefix;
  __shared__ int s_rem;
  const int64_t row = blockIdx.x;
  const int* st = a.state + row * 8;
  if (st[0] != 2) return;
  const int need = st[2];
  const int m = min(st[3], a.cand_cap);
  const uint32_t* ck = a.cand_key + row * a.cand_cap;
  const int32_t* ci = a.cand_idx + row * a.cand_cap;
  uint32_t* bm32 = (uint32_t*)(a.bitmap + row * a.bitmap_words);
  const int tid = threadIdx.x;
  if (need <= 0 || m <= 0) return;
  uint64_t thresh = 0;  // composite of the need-th largest (0: take all)
  if (need < m) {
    if (tid == 0) {
      s_prefix = 0;
      s_rem = need;
    }
    uint64_t pmask = 0;
    for (int shift = 56; shift >= 0; shift -= 8) {
      for (int i = tid; i < 256; i += 1024) h[i] = 0;
      __syncthreads();
      const uint64_t prefix = s_prefix;
      for (int i = tid; i < m; i += 1024) {
        const uint64_t comp = ((uint64_t)ck[i] << 32) | (uint32_t)(~ci[i]);
        if ((comp & pmask) == prefix) atomicAdd(&h[(comp >> shift) & 255], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        int rem = s_rem, acc = 0, dd = 255;
        for (; dd > 0; --dd) {
          if (acc + (int)h[dd] >= rem) break;
          acc += (int)h[dd];
        }
        s_rem = rem - acc;
        s_prefix = prefix | ((uint64_t)dd << shift);
      }
      pmask |= (uint64_t)255 << shift;
      __syncthreads();
    }
    thresh = s_prefix;
  }
  for (int i = tid; i < m; i += 1024) {
    const uint64_t comp = ((uint64_t)ck[i] << 32) | (uint32_t)(~ci[i]);
    if (comp >= thresh) {
      const int t = ci[i];
      atomicOr(&bm32[t >> 5], 1u << (t & 31));
    }
  }
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

// Ascending emission: bitmap tokens, then the window, then -1 padding.
// grid (rows), 1024 threads.
__global__ __launch_bounds__(1024) void k_sel_emit(SelArgs a) {
  __shared__ int lds16[16];
  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(a, row);
  int32_t* out = a.idx + row * a.S;
  const uint64_t* bm = a.bitmap + row * a.bitmap_words;
  const int tid = threadIdx.x;
  const int nwords = (ri.N + 63) >> 6;
  int base = 0;
  for (int w0 = 0; w0 < nwords; w0 += 1024) {
    const int w = w0 + tid;
    uint64_t bits = w < nwords ? bm[w] : 0ull;
    int total;
    int off = block_scan_1024(__popcll(bits), lds16, total);
    while (bits) {
      const int bit = __ffsll((long long)bits) - 1;
      bits &= bits - 1;
      const int p = base + off++;
      if (p < a.S) out[p] = 64 * w + bit;
    }
    base += total;
  }
  const int wlo = ri.pos - a.W + 1 < 0 ? 0 : ri.pos - a.W + 1;
  const int nw = ri.pos >= 0 ? ri.pos - wlo + 1 : 0;
  for (int j = tid; j < nw; j += 1024)
    if (base + j < a.S) out[base + j] = wlo + j;
  for (int j = base + nw + tid; j < a.S; j += 1024) out[j] = -1;
}

// ============================================================================ sparse attention
// grid (n_split, units = B * Hkv * C), 256 threads.  Rows: the Gp heads of
// KV head g for query c (RT_SA = Gp / 16 row tiles, at least 1).
template <int RT>
__global__ __launch_bounds__(NT) void k_sa_split(SaArgs a) {
  constexpr int TG = RT >= 4 ? 1 : 4 / RT;
  constexpr int RPW = RT >= 4 ? RT / 4 : 1;
  constexpr int BPW = 4 / TG;
  constexpr int WPT = 4 / TG;
  __shared__ TileLds lds;

  const int split = blockIdx.x;
  const int64_t unit = blockIdx.y;
  const int c = (int)(unit % a.C);
  const int g = (int)((unit / a.C) % a.Hkv);
  const int b = (int)(unit / ((int64_t)a.C * a.Hkv));
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int Lv = clamp_len(a.len, b, a.max_len);
  const int s_begin = split * a.split_slots;
  const int s_end = min(a.n_slots, s_begin + a.split_slots);
  const int tg = wave / WPT;
  const int rt0 = (wave % WPT) * RPW;

  // queries: heads h = 16 rt + (lane & 15) of query c
  uint4 q[RPW][4];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    const int h = 16 * (rt0 + rr) + (lane & 15);
    if (h < a.G) {
      const uint16_t* p = a.q + (((int64_t)b * a.C + c) * a.Hq + g * a.G + h) * HD + 8 * (lane >> 4);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) q[rr][kk] = *(const uint4*)(p + 32 * kk);
    } else {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) q[rr][kk] = make_uint4(0, 0, 0, 0);
    }
  }
  const int64_t kvoff = (int64_t)b * a.stride_b + (int64_t)g * a.stride_h;
  const uint16_t* Kbg = a.K + kvoff;
  const uint16_t* Vbg = a.V + kvoff;
  const int32_t* irow = a.idx + unit * a.idx_stride;
  const int cg = tid & 15;

  WaveState<RPW> st;
  st.init();
  int blk[BPW];
#pragma unroll
  for (int bi = 0; bi < BPW; ++bi) blk[bi] = tg * BPW + bi;

  auto gather = [&](int s0, int (&tok)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = s0 + row_of(tid, u);
      int t = s < s_end ? irow[s] : -1;
      if (t >= Lv) t = -1;
      tok[u] = t;
    }
  };
  TileRegs regs;
  int tok[4];
  if (s_begin < s_end) {
    gather(s_begin, tok);
    load_tile<true>(regs, Kbg, Vbg, a.stride_t, tok, cg);
  }
  for (int s0 = s_begin; s0 < s_end; s0 += TILE) {
    __syncthreads();
    store_tile<true>(lds, regs, tid);
    if (cg == 0) {
#pragma unroll
      for (int u = 0; u < 4; ++u) lds.tok[row_of(tid, u)] = tok[u];
    }
    __syncthreads();
    if (s0 + TILE < s_end) {
      gather(s0 + TILE, tok);
      load_tile<true>(regs, Kbg, Vbg, a.stride_t, tok, cg);
    }
    f32x4 S[BPW][RPW];
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) qk_block<RPW>(lds, blk[bi], q, S[bi], lane);
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) {
      int valid[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) valid[i] = lds.tok[16 * blk[bi] + 4 * (lane >> 4) + i] >= 0;
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr)
#pragma unroll
        for (int i = 0; i < 4; ++i) S[bi][rr][i] = valid[i] ? S[bi][rr][i] * a.c2 : -INFINITY;
    }
    softmax_pv<RPW, BPW>(st, lds, blk, S, lane);
  }
  const int nslot = a.n_split * TG;
  const int64_t slot_base_row = (unit * nslot + (int64_t)split * TG + tg) * (16 * RT);
  store_partial<RPW>(st, a.part_o, a.part_ml, slot_base_row, rt0, lane);
}

// ============================================================================ host launchers
#define HS2_LAUNCH(kernel, grid, block, shmem, stream, arg) \
  hipLaunchKernelGGL(kernel, grid, block, shmem, (hipStream_t)(stream), arg)

hipError_t launch_fa_split(const FaArgs& a, int RT, hipStream_t s) {
  dim3 grid(a.n_split, a.Hkv, a.B);
  switch (RT) {
    case 1: HS2_LAUNCH(k_fa_split<1>, grid, dim3(NT), 0, s, a); break;
    case 2: HS2_LAUNCH(k_fa_split<2>, grid, dim3(NT), 0, s, a); break;
    case 4: HS2_LAUNCH(k_fa_split<4>, grid, dim3(NT), 0, s, a); break;
    case 8: HS2_LAUNCH(k_fa_split<8>, grid, dim3(NT), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

size_t pool_smem_bytes(int RT, int C) {
  return KTILE_BYTES + (size_t)16 * RT * KPAD * sizeof(uint16_t) + (size_t)C * (NBINS / 2) * sizeof(uint32_t);
}

hipError_t launch_pool(const PoolArgs& a, int RT, hipStream_t s) {
  dim3 grid(a.n_split, a.Hkv, a.B);
  const size_t sm = pool_smem_bytes(RT, a.C);
  switch (RT) {
    case 1: HS2_LAUNCH(k_pool<1>, grid, dim3(NT), sm, s, a); break;
    case 2: HS2_LAUNCH(k_pool<2>, grid, dim3(NT), sm, s, a); break;
    case 4: HS2_LAUNCH(k_pool<4>, grid, dim3(NT), sm, s, a); break;
    case 8: HS2_LAUNCH(k_pool<8>, grid, dim3(NT), sm, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t set_pool_smem_limits() {
  // dynamic LDS above 64 KB must be allowed explicitly
  const int big = 160 * 1024;
  hipError_t e = hipSuccess;
  if (e == hipSuccess) e = hipFuncSetAttribute((const void*)k_pool<1>, hipFuncAttributeMaxDynamicSharedMemorySize, big);
  if (e == hipSuccess) e = hipFuncSetAttribute((const void*)k_pool<2>, hipFuncAttributeMaxDynamicSharedMemorySize, big);
  if (e == hipSuccess) e = hipFuncSetAttribute((const void*)k_pool<4>, hipFuncAttributeMaxDynamicSharedMemorySize, big);
  if (e == hipSuccess) e = hipFuncSetAttribute((const void*)k_pool<8>, hipFuncAttributeMaxDynamicSharedMemorySize, big);
  return e;
}

hipError_t launch_combine(const CombineArgs& a, int rows_per_unit, int64_t units, hipStream_t s) {
  HS2_LAUNCH(k_combine, dim3(rows_per_unit, (unsigned)units), dim3(HD), 0, s, a);
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
hipError_t launch_sel_threshold(const SelArgs& a, hipStream_t s) {
  HS2_LAUNCH(k_sel_threshold, dim3((unsigned)a.rows), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_sel_filter(const SelArgs& a, int nchunks, hipStream_t s) {
  HS2_LAUNCH(k_sel_filter, dim3(nchunks, (unsigned)a.rows), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_sel_resolve(const SelArgs& a, hipStream_t s) {
  HS2_LAUNCH(k_sel_resolve, dim3((unsigned)a.rows), dim3(1024), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_sel_emit(const SelArgs& a, hipStream_t s) {
  HS2_LAUNCH(k_sel_emit, dim3((unsigned)a.rows), dim3(1024), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sa_split(const SaArgs& a, int RT, hipStream_t s) {
  dim3 grid(a.n_split, (unsigned)((int64_t)a.B * a.Hkv * a.C));
  switch (RT) {
    case 1: HS2_LAUNCH(k_sa_split<1>, grid, dim3(NT), 0, s, a); break;
    case 2: HS2_LAUNCH(k_sa_split<2>, grid, dim3(NT), 0, s, a); break;
    case 4: HS2_LAUNCH(k_sa_split<4>, grid, dim3(NT), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hs2
