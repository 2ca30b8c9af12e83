// Device-side building blocks shared by the hybrid-block kernels (gfx950 only).
//
// Tile scheme: a workgroup of 256 threads (4 waves of 64) stages 64 cache rows
// at a time in LDS: K row-major (padded rows) and V transposed (Vt[d][row]),
// so that both MFMA operands of P.V can be read with plain LDS loads.
//
// MFMA lane layouts used (checked on gfx950):
//   16x16x32 bf16: lane l supplies A[l%16][8(l/16)+j] and B[8(l/16)+j][l%16],
//                  j = 0..7, and receives C[4(l/16)+i][l%16], i = 0..3;
//   16x16x16 bf16: same with 4(l/16)+j, j = 0..3, for A and B.
// Logits are computed as S^T = K . Q^T (tokens on MFMA rows, query rows on
// MFMA columns): lane l then holds four tokens 4(l/16)+i of query row l%16,
// which is exactly the A operand of the 16x16x16 product P . V.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs2 {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HD = 128;         // head dim served by these kernels
constexpr int TILE = 64;        // cache rows per LDS stage
constexpr int NT = 256;         // threads per workgroup
constexpr int KPAD = HD + 8;    // K / Q row stride in LDS (bf16): 272 B, conflict-free 16-B reads
constexpr int VPAD = TILE + 4;  // Vt row stride in LDS (bf16): 136 B
constexpr int NBINS = 2048;     // first-level radix bins of the pooled-score keys
constexpr int DIGIT_SHIFT = 18; // key >> 18 = 8 exponent bits + 5 mantissa bits
constexpr int DIGIT_BASE = 2240;// (exp 133, mant 31) -> bin 2047; P <= 64 < 128 always fits

struct TileLds {
  uint16_t k[TILE * KPAD];
  uint16_t vt[HD * VPAD];
  int32_t tok[TILE];  // token held by each tile row, -1 if none (gathered tiles)
};
constexpr size_t KTILE_BYTES = sizeof(uint16_t) * TILE * KPAD;  // the K part alone

__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16, round to nearest even (inputs are finite here)
__device__ inline uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ inline f32x4 mfma_k32(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                 0, 0, 0);
}
__device__ inline f32x4 mfma_k16(const uint2& a, const uint2& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4, a), __builtin_bit_cast(i16x4, b), c,
                                                   0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Ordered key of a pooled score: IEEE bits of a non-negative float are
// monotone as unsigned integers; values below FLT_MIN count as +0.
__device__ inline uint32_t score_key(float p) {
  return p < 1.17549435e-38f ? 0u : __float_as_uint(p);
}
__device__ inline int score_digit(uint32_t key) {
  int d = (int)(key >> DIGIT_SHIFT) - DIGIT_BASE;
  return d < 0 ? 0 : (d >= NBINS ? NBINS - 1 : d);
}

// ---------------------------------------------------------------- tile staging
// Thread tid owns four 16-byte chunks of the 64 x 16 chunk grid of a tile:
// column group cg = tid & 15, rows row_of(tid, u), u = 0..3.  Rows come in
// adjacent pairs (u = 0, 1 and u = 2, 3) so V can be stored transposed two
// tokens (one 32-bit word) at a time.  Every 16 lanes read one full 256-byte
// cache row: loads are fully coalesced.
__device__ inline int row_of(int tid, int u) { return 2 * (tid >> 4) + (u & 1) + 32 * (u >> 1); }

struct TileRegs {
  uint4 k[4];
  uint4 v[4];
};

// Load the K and V rows of tokens tok[u] (tok < 0: zeros) of one (b, g) cache.
template <bool WITH_V>
__device__ inline void load_tile(TileRegs& r, const uint16_t* __restrict__ Kbg, const uint16_t* __restrict__ Vbg,
                                 int64_t stride_t, const int (&tok)[4], int cg) {
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (tok[u] >= 0) {
      const int64_t off = (int64_t)tok[u] * stride_t + cg * 8;
      r.k[u] = *(const uint4*)(Kbg + off);
      if (WITH_V) r.v[u] = *(const uint4*)(Vbg + off);
    } else {
      r.k[u] = make_uint4(0, 0, 0, 0);
      if (WITH_V) r.v[u] = make_uint4(0, 0, 0, 0);
    }
  }
}

template <bool WITH_V>
__device__ inline void store_tile(TileLds& s, const TileRegs& r, int tid) {
  const int cg = tid & 15;
#pragma unroll
  for (int u = 0; u < 4; ++u) *(uint4*)&s.k[row_of(tid, u) * KPAD + cg * 8] = r.k[u];
  if (WITH_V) {
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      const int row = row_of(tid, 2 * pr);  // even row; row + 1 is its pair
      const uint32_t* a = (const uint32_t*)&r.v[2 * pr];
      const uint32_t* b = (const uint32_t*)&r.v[2 * pr + 1];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        // word w of a chunk holds elements d = cg*8 + 2w (low half) and +1 (high half)
        const uint32_t lo = (a[w] & 0xFFFFu) | (b[w] << 16);
        const uint32_t hi = (a[w] >> 16) | (b[w] & 0xFFFF0000u);
        *(uint32_t*)&s.vt[(cg * 8 + 2 * w) * VPAD + row] = lo;
        *(uint32_t*)&s.vt[(cg * 8 + 2 * w + 1) * VPAD + row] = hi;
      }
    }
  }
}

// ---------------------------------------------------------------- wave-level attention state
// One wave, RPW row tiles of 16 query rows.  m: running max of log2-domain
// logits of row (lane & 15) (same in all four lane groups); l: this lane's
// share of the running sum; o: unnormalised output rows 4(lane/16)+i,
// columns 16*nb + (lane & 15).
template <int RPW>
struct WaveState {
  float m[RPW];
  float l[RPW];
  f32x4 o[RPW][8];
  __device__ inline void init() {
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      m[r] = -INFINITY;
      l[r] = 0.f;
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) o[r][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

// Logits of the 16 tile rows of block `blk` against RPW row tiles of queries
// (B operands in registers): S[rr][i] = <K[16 blk + 4(lane/16) + i], Q[row lane&15]>.
template <int RPW>
__device__ inline void qk_block(const TileLds& s, int blk, const uint4 (&q)[RPW][4], f32x4 (&S)[RPW], int lane) {
  const uint16_t* kp = &s.k[(16 * blk + (lane & 15)) * KPAD + 8 * (lane >> 4)];
  uint4 a[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) a[kk] = *(const uint4*)(kp + 32 * kk);
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc = mfma_k32(a[kk], q[rr][kk], acc);
    S[rr] = acc;
  }
}

// Online-softmax update with BPW blocks of log2-domain logits (masked = -inf),
// then O += P . V over those blocks.
template <int RPW, int BPW>
__device__ inline void softmax_pv(WaveState<RPW>& st, const TileLds& s, const int (&blk)[BPW],
                                  f32x4 (&S)[BPW][RPW], int lane) {
  uint2 pa[BPW][RPW];
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    float mx = -INFINITY;
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi)
#pragma unroll
      for (int i = 0; i < 4; ++i) mx = fmaxf(mx, S[bi][rr][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(st.m[rr], mx);
    const float msub = (mnew == -INFINITY) ? 0.f : mnew;
    const float alpha = fast_exp2(st.m[rr] - msub);  // m = -inf -> 0; unchanged max -> 1
    st.m[rr] = mnew;
    float psum = 0.f;
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) {
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = fast_exp2(S[bi][rr][i] - msub);
        psum += p[i];
      }
      pa[bi][rr].x = f32_to_bf16_bits(p[0]) | (f32_to_bf16_bits(p[1]) << 16);
      pa[bi][rr].y = f32_to_bf16_bits(p[2]) | (f32_to_bf16_bits(p[3]) << 16);
    }
    st.l[rr] = st.l[rr] * alpha + psum;
    if (__ballot(alpha != 1.f)) {
      float a4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a4[i] = __shfl(alpha, 4 * (lane >> 4) + i);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) st.o[rr][nb][i] *= a4[i];
    }
  }
#pragma unroll
  for (int bi = 0; bi < BPW; ++bi) {
    const uint16_t* vp = &s.vt[(lane & 15) * VPAD + 16 * blk[bi] + 4 * (lane >> 4)];
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      const uint2 vb = *(const uint2*)(vp + 16 * nb * VPAD);
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k16(pa[bi][rr], vb, st.o[rr][nb]);
    }
  }
}

// Write one wave's partial (m, l, O) for its RPW row tiles.
template <int RPW>
__device__ inline void store_partial(const WaveState<RPW>& st, float* __restrict__ part_o,
                                     float* __restrict__ part_ml, int64_t slot_base_row, int rt0, int lane) {
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    float l = st.l[rr];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int64_t row0 = slot_base_row + 16 * (rt0 + rr);
    if (lane < 16) {
      part_ml[(row0 + lane) * 2] = st.m[rr];
      part_ml[(row0 + lane) * 2 + 1] = l;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* dst = part_o + (row0 + 4 * (lane >> 4) + i) * HD + (lane & 15);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) dst[16 * nb] = st.o[rr][nb][i];
    }
  }
}

}  // namespace hs2
