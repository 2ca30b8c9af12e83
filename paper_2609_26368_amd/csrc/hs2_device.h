// Device-side building blocks shared by the hybrid-block kernels (gfx950 only).
//
// Staging: cache rows go global -> LDS by 16-byte direct-to-LDS loads (no
// register staging), row-major, 16-byte chunks swizzled by the row index so
// that the MFMA K-operand reads and the transposing V reads
// (ds_read_b64_tr_b16) are free of bank conflicts without padding; E4M3
// rows are staged raw (swizzled too); K is converted in registers (or into
// a bf16 tile of the same layout when several waves share it), V is read
// raw by an 8-bit transposing read and converted in registers.
//
// MFMA lane layouts used (checked on gfx950):
//   16x16x32 bf16: lane l supplies A[l%16][8(l/16)+j] and B[8(l/16)+j][l%16],
//                  j = 0..7, and receives C[4(l/16)+i][l%16], i = 0..3;
//   16x16x16 bf16: same with 4(l/16)+j, j = 0..3, for A and B.
// Logits are computed as S^T = K . Q^T (tokens on MFMA rows, query rows on
// MFMA columns): lane l then holds four tokens 4(l/16)+i of query row l%16,
// which is exactly the A operand of the 16x16x16 product P . V (two such
// blocks side by side: the A operand of a 16x16x32 product).  The logits'
// k slots carry the head dims in the order of q_koff / k_chunk.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hs2 {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int HD = 128;         // head dim of the workgroup kernel; the ring kernels take theirs as a parameter
constexpr int TILE = 64;        // cache rows per LDS stage of the workgroup kernel
constexpr int NT = 256;         // threads per workgroup of the score and histogram kernels
constexpr int SEL_CHUNK = 4096;  // tokens per workgroup of the selection scans
constexpr int NBINS = 1024;     // first-level radix bins of the pooled-score keys
constexpr int DIGIT_SHIFT = 19; // key >> 19 = 8 exponent bits + 4 mantissa bits (1/16 binade)
constexpr int DIGIT_BASE = 1120;// (exp 133, mant 15) -> bin 1023: 64 binades below 128 > P;
                                // P < 2^-56 all fall into bin 0

__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16, round to nearest even (inputs are finite here)
__device__ inline uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two fp32 -> packed bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32)
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
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
// First-level radix digit (histogram bin) of a score: its key's top bits
// clamped to the NBINS bins.  Taken straight from the float bits with one
// clamp: a value below FLT_MIN (or negative) lands in bin 0 like its key
// +0, so this equals the digit of score_key(p) for every input but NaNs
// with the sign bit set (bin 0 here; no score is NaN).  Every histogram and
// filter derives its bins with this one function.
__device__ inline int score_digit(float p) {
  const int x = __float_as_int(p) >> DIGIT_SHIFT;  // arithmetic shift: negative values stay negative
  return min(max(x, DIGIT_BASE), DIGIT_BASE + NBINS - 1) - DIGIT_BASE;
}

// ---------------------------------------------------------------- wave-level attention state
// One wave, RPW row tiles of 16 query rows, for row (lane & 15) (same in all
// four lane groups): m is the reference the probabilities exp2(s - m) are
// taken against, mt the true running maximum of the log2-domain logits; l is
// this lane's share of the running sum; o holds the unnormalised output rows
// 4(lane/16)+i, columns 16*nb + (lane & 15).
// x combined with its value in lane ^ 16 (^ 32) through gfx950's VALU lane
// swaps instead of an LDS permute: swapping a register with itself leaves
// each lane's pair {x[lane], x[lane ^ 16]} in the two result registers, so
// max and sum are identical in both lanes of a pair.
__device__ inline float2 lane_pair16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float2 lane_pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float max_xor16(float x) { const float2 p = lane_pair16(x); return fmaxf(p.x, p.y); }
__device__ inline float max_xor32(float x) { const float2 p = lane_pair32(x); return fmaxf(p.x, p.y); }
__device__ inline float sum_xor16(float x) { const float2 p = lane_pair16(x); return p.x + p.y; }
__device__ inline float sum_xor32(float x) { const float2 p = lane_pair32(x); return p.x + p.y; }

template <int RPW, int HDIM = HD>
struct WaveState {
  static constexpr int NBC = HDIM / 16;  // 16-column blocks of O
  float m[RPW];   // reference maximum the probabilities are taken against
  float mt[RPW];  // true running maximum (for the reported statistics)
  float l[RPW];
  f32x4 o[RPW][NBC];
  __device__ inline void init() {
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      m[r] = -INFINITY;
      mt[r] = -INFINITY;
      l[r] = 0.f;
#pragma unroll
      for (int nb = 0; nb < NBC; ++nb) o[r][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }
};

// Online-softmax update of a wave's state with BPW blocks of log2-domain
// logits (masked = -inf); returns the bf16 probabilities as P.V A operands.
// The reference maximum m is raised only when a logit exceeds it by more
// than LAZY_MARGIN, so probabilities stay <= 2^LAZY_MARGIN and the
// accumulators are rescaled rarely; the true maximum is tracked in mt.
constexpr float LAZY_MARGIN = 8.f;

// bf16 probabilities of BPW 16-token blocks x RPW row tiles in the layout of
// the P.V A operands: with K32, blocks 2 bp and 2 bp + 1 share one 16x16x32
// operand w[bp] (x, y: block 2 bp; z, w: block 2 bp + 1); otherwise block bi
// is the 16x16x16 operand h[bi].  Written straight into this layout, the
// fragments stay in registers.
template <int BPW, int RPW, bool K32 = BPW % 2 == 0>
struct PFrags {
  static_assert(!K32 || BPW % 2 == 0, "paired blocks");
  uint4 w[K32 ? BPW / 2 : 1][RPW];
  uint2 h[K32 ? 1 : BPW][RPW];
  __device__ inline void set(int bi, int rr, uint32_t lo, uint32_t hi) {
    if constexpr (K32) {
      if (bi & 1) {
        w[bi >> 1][rr].z = lo;
        w[bi >> 1][rr].w = hi;
      } else {
        w[bi >> 1][rr].x = lo;
        w[bi >> 1][rr].y = hi;
      }
    } else {
      h[bi][rr] = make_uint2(lo, hi);
    }
  }
};

template <int RPW, int BPW, int HDIM, bool K32>
__device__ inline void online_softmax(WaveState<RPW, HDIM>& st, f32x4 (&S)[BPW][RPW], PFrags<BPW, RPW, K32>& pf,
                                      int lane) {
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    float mx = -INFINITY;
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi)
      mx = fmaxf(mx, fmaxf(fmaxf(S[bi][rr][0], S[bi][rr][1]), fmaxf(S[bi][rr][2], S[bi][rr][3])));
    mx = max_xor32(max_xor16(mx));
    st.mt[rr] = fmaxf(st.mt[rr], mx);
    if (__ballot(mx > st.m[rr] + LAZY_MARGIN)) {
      const float mnew = fmaxf(st.m[rr], mx);
      const float alpha = mnew == -INFINITY ? 1.f : fast_exp2(st.m[rr] - mnew);  // m = -inf -> 0
      st.m[rr] = mnew;
      st.l[rr] *= alpha;
      float a4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a4[i] = __shfl(alpha, 4 * (lane >> 4) + i);
#pragma unroll
      for (int nb = 0; nb < WaveState<RPW, HDIM>::NBC; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) st.o[rr][nb][i] *= a4[i];
    }
    const float msub = st.m[rr] == -INFINITY ? 0.f : st.m[rr];
    float psum = 0.f;
#pragma unroll
    for (int bi = 0; bi < BPW; ++bi) {
      float p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = fast_exp2(S[bi][rr][i] - msub);
        psum += p[i];
      }
      pf.set(bi, rr, pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]));
    }
    st.l[rr] += psum;
  }
}

// Write one wave's partial for its RPW row tiles: (m ref, l, m true, 0) and O
// (rows of HDIM floats).
template <int RPW, int HDIM>
__device__ inline void store_partial(const WaveState<RPW, HDIM>& st, float* __restrict__ part_o,
                                     float* __restrict__ part_ml, int64_t slot_base_row, int rt0, int lane) {
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    float l = st.l[rr];
    l = sum_xor32(sum_xor16(l));
    const int64_t row0 = slot_base_row + 16 * (rt0 + rr);
    if (lane < 16) *(float4*)(part_ml + (row0 + lane) * 4) = make_float4(st.m[rr], l, st.mt[rr], 0.f);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float* dst = part_o + (row0 + 4 * (lane >> 4) + i) * HDIM + (lane & 15);
#pragma unroll
      for (int nb = 0; nb < WaveState<RPW, HDIM>::NBC; ++nb) dst[16 * nb] = st.o[rr][nb][i];
    }
  }
}


// ---------------------------------------------------------------- direct-to-LDS staging (swizzled)
// One stage holds TILE cache rows of K then TILE rows of V, 256 bytes each,
// row-major; the 16-byte chunk c of row r sits at position c ^ stage_swz(r)
// of the row.  stage_swz(r) mod 8 is a permutation of rows 0-7 and of rows
// 8-15, so one chunk of 8 consecutive rows (the MFMA K-operand reads) lands
// in 8 distinct slots of a 128-byte window; its bits 1-2 are r & 3, so the
// transposing V reads (4 rows x chunks 2m, 2m + 1) land in 8 distinct slots
// as well; and it is a permutation of all 16 rows.  With it both reads were
// measured free of bank conflicts (with c ^ (r & 15) the V reads were
// 2-way).  A wave's 16-byte direct LDS load writes 64 consecutive 16-byte
// slots (lane order): load n = 4 * wave + u fills slots 64 n + lane, i.e.
// row 4 n + lane / 16, position lane % 16.
__device__ __host__ constexpr int stage_swz(int r) {
  return ((r & 3) << 1) | (((r >> 2) & 1) << 3) | (((r >> 2) ^ (r >> 3)) & 1);
}
constexpr int STAGE_ROW_BYTES = HD * 2;
constexpr int STAGE_KV_BYTES = TILE * STAGE_ROW_BYTES;  // 16 KB
constexpr int STAGE_BYTES = 2 * STAGE_KV_BYTES;         // K + V
constexpr int FA_STAGES = 4;

typedef short i16x4_lds __attribute__((ext_vector_type(4)));

// NW waves share the loads of a stage: LPW = 16 / NW loads of 1 KB per
// matrix per wave; load n = LPW * wave + u fills rows 4 n .. 4 n + 3.
template <int NW>
__device__ inline int stage_row(int wave, int u, int lane) {
  return 4 * ((16 / NW) * wave + u) + (lane >> 4);
}

// One 16-byte-per-lane direct LDS load: lane i's 16 bytes from `src` land at
// LDS byte address lds_base + 16 i.  Issued as inline assembly so that the
// compiler does not guard every later LDS read with a wait for all
// outstanding loads; the caller waits explicitly (wait_stage_loads) and
// then synchronises the workgroup before reading the stage.
__device__ inline void dma16(const void* src, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds_base) : "memory");
}

// The same load with the non-temporal hint when NTH: for rows read once, they
// stream past the caches instead of evicting lines a later pass reads again.
template <bool NTH>
__device__ inline void dma16_p(const void* src, uint32_t lds_base) {
  if constexpr (NTH)
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" : : "v"(src), "s"(lds_base) : "memory");
  else
    dma16(src, lds_base);
}

// The same load from a wave-uniform base (scalar registers) plus this lane's
// 32-bit byte offset: no per-lane 64-bit address arithmetic.
__device__ inline const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
template <bool NTH>
__device__ inline void dma16_s(const void* sbase, uint32_t voff, uint32_t lds_base) {
  sbase = uniform_ptr(sbase);  // (free where the base is already scalar)
  if constexpr (NTH)
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1 nt" : : "v"(voff), "s"(sbase), "s"(lds_base) : "memory");
  else
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff), "s"(sbase), "s"(lds_base) : "memory");
}

__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Issue this wave's share of one stage: rows tok[u] (u < 16 / NW) of K and V.
template <int NW>
__device__ inline void issue_stage_loads(unsigned char* stage, const uint16_t* Kbg, const uint16_t* Vbg,
                                         int64_t stride_t, const int* tok, int wave, int lane) {
  constexpr int LPW = 16 / NW;
  const uint32_t base = lds_addr(stage);
#pragma unroll
  for (int u = 0; u < LPW; ++u) {
    const int n = LPW * wave + u;
    const int r = stage_row<NW>(wave, u, lane);
    const int c = (lane & 15) ^ stage_swz(r);
    const int64_t off = (int64_t)tok[u] * stride_t + 8 * c;
    dma16(Kbg + off, __builtin_amdgcn_readfirstlane(base + 1024 * n));
    dma16(Vbg + off, __builtin_amdgcn_readfirstlane(base + STAGE_KV_BYTES + 1024 * n));
  }
}

// s_waitcnt until at most `tiles` stages of this wave's loads (2 * 16 / NW
// each) are outstanding.  gfx9 encoding: vmcnt = bits [3:0] | [15:14];
// expcnt [6:4] and lgkmcnt [11:8] stay at their maxima.
template <int NW>
__device__ inline void wait_stage_loads(int tiles) {
  if (NW == 4) {
    if (tiles <= 0) __builtin_amdgcn_s_waitcnt(0x0F70);       // vmcnt(0)
    else if (tiles == 1) __builtin_amdgcn_s_waitcnt(0x0F78);  // vmcnt(8)
    else __builtin_amdgcn_s_waitcnt(0x4F70);                  // vmcnt(16)
  } else {
    if (tiles <= 0) __builtin_amdgcn_s_waitcnt(0x0F70);       // vmcnt(0)
    else if (tiles == 1) __builtin_amdgcn_s_waitcnt(0x0F74);  // vmcnt(4)
    else __builtin_amdgcn_s_waitcnt(0x0F78);                  // vmcnt(8)
  }
}

// The k order of the logits MFMAs (16x16x32): for MFMA kk, lane group
// j = lane / 16 holds the 8 head dims 64 (kk / 2) + 16 j + 8 (kk % 2) .. + 7,
// in the K operands and the query operands alike.  So MFMAs 2 i and 2 i + 1
// of a lane together cover one 16-dim run, which one 16-byte read of an
// E4M3 row supplies; a bf16 row supplies it as two 16-byte chunks.
__device__ inline int q_koff(int kk, int lane) { return 64 * (kk >> 1) + 16 * (lane >> 4) + 8 * (kk & 1); }
__device__ inline int k_chunk(int kk, int lane) { return 8 * (kk >> 1) + 2 * (lane >> 4) + (kk & 1); }

// Logits S^T = K . Q^T of the 16 staged rows of block blk; rows of 64 NKK
// bytes (head dim 32 NKK), swizzled chunks.
template <int RPW, int NKK>
__device__ inline void qk_block_swz(const unsigned char* stg, int blk, const uint4 (&q)[RPW][NKK], f32x4 (&S)[RPW],
                                    int lane) {
  const int row = 16 * blk + (lane & 15);
  const unsigned char* rp = stg + row * (64 * NKK);
  uint4 a4[NKK];
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk) a4[kk] = *(const uint4*)(rp + 16 * (k_chunk(kk, lane) ^ stage_swz(row)));
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) acc = mfma_k32(a4[kk], q[rr][kk], acc);
    S[rr] = acc;
  }
}

// V operand of P.V for block blk, columns 16 nb .. 16 nb + 15 (16x16x16 B layout),
// read transposed from the row-major stage.
__device__ inline uint2 v_operand_tr(const unsigned char* stg, int blk, int nb, int lane) {
  const int kq = lane & 15;
  const int row = 16 * blk + 4 * (lane >> 4) + (kq >> 2);
  const int col = 16 * nb + 4 * (kq & 3);
  const int pos = (col >> 3) ^ stage_swz(row);
  const unsigned char* p = stg + STAGE_KV_BYTES + row * STAGE_ROW_BYTES + 16 * pos + 2 * (col & 7);
  const i16x4_lds v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4_lds*)(p));
  return __builtin_bit_cast(uint2, v);
}

template <int RPW, int BPW>
__device__ inline void softmax_pv_swz(WaveState<RPW>& st, const unsigned char* stg, const int (&blk)[BPW],
                                      f32x4 (&S)[BPW][RPW], int lane) {
  PFrags<BPW, RPW, false> pf;
  online_softmax(st, S, pf, lane);
#pragma unroll
  for (int bi = 0; bi < BPW; ++bi) {
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      const uint2 vb = v_operand_tr(stg, blk[bi], nb, lane);
#pragma unroll
      for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k16(pf.h[bi][rr], vb, st.o[rr][nb]);
    }
  }
}


// ---------------------------------------------------------------- wave-private staging
// A one-wave workgroup streams its own token range through a private ring of
// NS stages, each holding TW rows of K then TW rows of V (swizzled as above).
// No workgroup barrier: the wave only waits for its own direct LDS loads.
constexpr int vmcnt_enc(int n) { return (n & 15) | ((n >> 4) << 14) | 0x0F70; }

// ---------------------------------------------------------------- FP8 cache rows
// An FP8 (OCP E4M3) cache row is HDIM bytes.  Rows are staged raw (row-major)
// by the same 16-byte direct LDS loads -- a 1 KB load covers 1024 / HDIM
// rows -- and converted into the bf16 stage layout above, so every bf16
// operand read is shared by both cache formats.

// Four E4M3 values (the bytes of w, low first) -> four bf16 in two packed
// words, exactly (every E4M3 value is a bf16 value): gfx950's scaled
// conversion with scale 1 of bytes 0-1, then of bytes 2-3 shifted down.
// Through the compiler builtin (its low-word form: the word-select form
// produced the upper pair as a copy of the lower on this toolchain), not
// inline assembly: the compiler then keeps the wait states an MFMA needs
// before a VALU instruction overwrites one of its source registers, which
// it does not do around inline assembly.
__device__ inline uint32_t e4m3x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false));
}
__device__ inline uint2 e4m3x4_to_bf16x4(uint32_t w) {
  return make_uint2(e4m3x2_to_bf16x2(w), e4m3x2_to_bf16x2(w >> 16));
}

// Raw E4M3 rows of RB bytes are staged swizzled too: chunk c of row r at
// position c ^ raw_swz<RB>(r), r modulo the chunks of a row, so that the
// 16-byte K-operand reads (one chunk of each of 16 rows) spread over all
// chunk slots (measured free of bank conflicts, as are the row-contiguous
// conversion reads).
template <int RB>
__device__ __host__ constexpr int raw_swz(int r) {
  return r & (RB / 16 - 1);
}

// Operands of the logits MFMAs 2 i and 2 i + 1 (16x16x32, row `row`) from a
// raw E4M3 stage, converted to bf16 in registers: one 16-byte chunk
// c = lane / 16 + 4 i (head dims 16 c .. 16 c + 15), its first 8 values for
// MFMA 2 i and its last 8 for MFMA 2 i + 1 (the order of q_koff).
template <int RB>
__device__ inline void k_operands_e4m3(const unsigned char* raw, int row, int i, int lane, uint4& a0, uint4& a1) {
  const int c = (lane >> 4) + 4 * i;
  const uint4 v = *(const uint4*)(raw + row * RB + 16 * (c ^ raw_swz<RB>(row)));
  const uint2 x = e4m3x4_to_bf16x4(v.x), y = e4m3x4_to_bf16x4(v.y);
  const uint2 z = e4m3x4_to_bf16x4(v.z), w = e4m3x4_to_bf16x4(v.w);
  a0 = make_uint4(x.x, x.y, y.x, y.y);
  a1 = make_uint4(z.x, z.y, w.x, w.y);
}

// Logits of the 16 rows of block blk of a raw E4M3 stage against RPW row
// tiles of queries (as qk_block_swz, K converted in registers).
template <int RPW, int RB, int NKK>
__device__ inline void qk_block_e4m3(const unsigned char* raw, int blk, const uint4 (&q)[RPW][NKK], f32x4 (&S)[RPW],
                                     int lane) {
  const int row = 16 * blk + (lane & 15);
  uint4 a4[NKK];
#pragma unroll
  for (int i = 0; i < NKK / 2; ++i) k_operands_e4m3<RB>(raw, row, i, lane, a4[2 * i], a4[2 * i + 1]);
#pragma unroll
  for (int rr = 0; rr < RPW; ++rr) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) acc = mfma_k32(a4[kk], q[rr][kk], acc);
    S[rr] = acc;
  }
}

// LDS of a full-attention ring kernel: per token group an NS-stage ring of
// TW K rows and TW V rows (bf16: 2 hd bytes a row; E4M3: hd bytes, plus
// converted bf16 K and V tiles when the group has several waves); at least
// the end-of-split merge of TGW groups.
__device__ __host__ constexpr int fa_ring_group_bytes(int nwv, int tw, int ns, bool kv8, int hd) {
  return ns * 2 * tw * (kv8 ? hd : 2 * hd) + (kv8 && nwv > 1 ? 2 * tw * 2 * hd : 0);
}
__device__ __host__ constexpr int fa_ring_merge_bytes(int rt, int tgw, int hd) {
  return tgw > 1 ? tgw * 16 * rt * 16 + (tgw - 1) * 16 * rt * hd * 4 : 0;
}
__device__ __host__ constexpr int fa_ring_lds_bytes(int rt, int nwv, int tw, int ns, int tgw, bool kv8, int hd) {
  return tgw * fa_ring_group_bytes(nwv, tw, ns, kv8, hd) > fa_ring_merge_bytes(rt, tgw, hd)
             ? tgw * fa_ring_group_bytes(nwv, tw, ns, kv8, hd)
             : fa_ring_merge_bytes(rt, tgw, hd);
}

// Convert NR staged E4M3 rows (raw, HDIM bytes each, chunk c of row r at
// position c ^ raw_swz(r)) into bf16 stage rows at stg (2 HDIM bytes; chunk c
// of row r at position c ^ stage_swz(r)); threads tid of NTHR.  A job is one
// 16-byte raw piece p of row r: 16 values, bf16 chunks 2 p and 2 p + 1.
// Eight consecutive jobs take pieces 4 m' .. 4 m' + 3 of rows r and r + 4 of
// an 8-row block (r < 4 within it): those rows' stage_swz differ in bit 0,
// so each of the two stores of 8 lanes covers 8 distinct 16-byte slots of a
// 128-byte window, and so does the raw read.
template <int NR, int NTHR, int HDIM>
__device__ inline void convert_rows_e4m3(const unsigned char* raw, unsigned char* stg, int tid) {
  constexpr int PPR = HDIM / 16;  // raw pieces per row
  constexpr int JOBS = NR * PPR;
  static_assert(NR % 8 == 0 && PPR % 4 == 0, "8-row blocks, 4-piece quads");
#pragma unroll
  for (int k = 0; k < (JOBS + NTHR - 1) / NTHR; ++k) {
    const int j = tid + k * NTHR;
    if (JOBS % NTHR == 0 || j < JOBS) {
      const int jb = j % (8 * PPR), m = jb >> 3;
      const int r = 8 * (j / (8 * PPR)) + (m & 3) + 4 * ((jb >> 2) & 1);
      const int p = 4 * (m >> 2) + (jb & 3);
      const uint4 v = *(const uint4*)(raw + r * HDIM + 16 * (p ^ raw_swz<HDIM>(r)));
      const uint2 a = e4m3x4_to_bf16x4(v.x), b = e4m3x4_to_bf16x4(v.y);
      const uint2 c = e4m3x4_to_bf16x4(v.z), d = e4m3x4_to_bf16x4(v.w);
      unsigned char* rp = stg + r * (2 * HDIM);
      *(uint4*)(rp + 16 * ((2 * p) ^ stage_swz(r))) = make_uint4(a.x, a.y, b.x, b.y);
      *(uint4*)(rp + 16 * ((2 * p + 1) ^ stage_swz(r))) = make_uint4(c.x, c.y, d.x, d.y);
    }
  }
}

// s_waitcnt vmcnt(per_stage * stages) for stages in [0, 5] (larger values
// wait as for 5; counts above the 6-bit field wait for 63: both only wait
// longer than needed)
constexpr int vmcnt_enc_sat(int n) { return vmcnt_enc(n > 63 ? 63 : n); }
template <int PER_STAGE>
__device__ inline void wait_ring(int stages) {
  switch (stages) {
    case 0: __builtin_amdgcn_s_waitcnt(vmcnt_enc(0)); break;
    case 1: __builtin_amdgcn_s_waitcnt(vmcnt_enc_sat(PER_STAGE)); break;
    case 2: __builtin_amdgcn_s_waitcnt(vmcnt_enc_sat(2 * PER_STAGE)); break;
    case 3: __builtin_amdgcn_s_waitcnt(vmcnt_enc_sat(3 * PER_STAGE)); break;
    case 4: __builtin_amdgcn_s_waitcnt(vmcnt_enc_sat(4 * PER_STAGE)); break;
    default: __builtin_amdgcn_s_waitcnt(vmcnt_enc_sat(5 * PER_STAGE)); break;
  }
}

// V operand of P.V for block blk, columns 16 nb .. 16 nb + 15, read
// transposed from the row-major swizzled V rows (2 HDIM bytes) at `vbase`.
template <int HDIM>
__device__ inline uint2 v_operand_tr_at(const unsigned char* vbase, int blk, int nb, int lane) {
  const int kq = lane & 15;
  const int row = 16 * blk + 4 * (lane >> 4) + (kq >> 2);
  const int col = 16 * nb + 4 * (kq & 3);
  const int pos = (col >> 3) ^ stage_swz(row);
  const unsigned char* p = vbase + row * (2 * HDIM) + 16 * pos + 2 * (col & 7);
  const i16x4_lds v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4_lds*)(p));
  return __builtin_bit_cast(uint2, v);
}


// V operands of P.V straight from raw E4M3 V rows (RB bytes, chunk c of row
// r at c ^ raw_swz(r)) by gfx950's 8-bit transposing LDS read: in each
// 16-lane group, lane pair p supplies 8 bytes of one row and lane q receives
// byte q of the group's 16-byte columns, i.e. one head dim of the 8 rows
// (checked on the device).  Each lane pair names the row it wants, so the 8
// tokens come in the k order of the P fragments: for a pair of 16-token
// blocks, the lane group's 4 tokens of block 2 bp, then its 4 of block
// 2 bp + 1 (as v_operand_tr_at twice); the 8 values are then converted to
// bf16 in registers (exact).
template <int RB>
__device__ inline uint2 ds_read_tr8(const unsigned char* raw_v, int row, int nb, int lane) {
  typedef int v2i __attribute__((ext_vector_type(2)));
  const unsigned char* p = raw_v + row * RB + 16 * (nb ^ raw_swz<RB>(row)) + 8 * (lane & 1);
  const v2i r = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i*)(p));
  return make_uint2((uint32_t)r.x, (uint32_t)r.y);
}
// head dims 16 nb .. 16 nb + 15 of blocks 2 bp, 2 bp + 1 (16x16x32 B operand)
template <int RB>
__device__ inline uint4 v_operand_e4m3_pair(const unsigned char* raw_v, int bp, int nb, int lane) {
  const int g = lane >> 4, r = (lane & 15) >> 1;
  const int row = 32 * bp + 16 * (r >> 2) + 4 * g + (r & 3);
  const uint2 x = ds_read_tr8<RB>(raw_v, row, nb, lane);
  const uint2 lo = e4m3x4_to_bf16x4(x.x), hi = e4m3x4_to_bf16x4(x.y);
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}
// head dims 16 nb .. 16 nb + 15 of block bi (16x16x16 B operand: the lane
// group's 4 tokens; the lane pairs 4 .. 7 repeat rows 0 .. 3)
template <int RB>
__device__ inline uint2 v_operand_e4m3(const unsigned char* raw_v, int bi, int nb, int lane) {
  const int g = lane >> 4, r = (lane & 15) >> 1;
  const uint2 x = ds_read_tr8<RB>(raw_v, 16 * bi + 4 * g + (r & 3), nb, lane);
  return e4m3x4_to_bf16x4(x.x);
}

// O += P . V for the NB 16-token blocks of a raw E4M3 V tile (RB-byte rows).
template <int RPW, int NB, int HDIM, int RB>
__device__ inline void pv_tile_e4m3(WaveState<RPW, HDIM>& st, const PFrags<NB, RPW>& pf, const unsigned char* raw_v,
                                    int lane) {
  if constexpr (NB % 2 == 0) {
#pragma unroll
    for (int bp = 0; bp < NB / 2; ++bp)
#pragma unroll
      for (int nb = 0; nb < HDIM / 16; ++nb) {
        const uint4 vb = v_operand_e4m3_pair<RB>(raw_v, bp, nb, lane);
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k32(pf.w[bp][rr], vb, st.o[rr][nb]);
      }
  } else {
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
      for (int nb = 0; nb < HDIM / 16; ++nb) {
        const uint2 vb = v_operand_e4m3<RB>(raw_v, bi, nb, lane);
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k16(pf.h[bi][rr], vb, st.o[rr][nb]);
      }
  }
}

// O += P . V for the NB 16-token blocks of a staged tile (V rows swizzled at
// vbase).  With an even NB two blocks share one 16x16x32 product: k slots
// 8 (lane / 16) + j hold the lane group's 4 tokens of block 2 bp, then its 4
// of block 2 bp + 1, in the P fragments and the transposed V reads alike.
template <int RPW, int NB, int HDIM>
__device__ inline void pv_tile(WaveState<RPW, HDIM>& st, const PFrags<NB, RPW>& pf, const unsigned char* vbase,
                               int lane) {
  if constexpr (NB % 2 == 0) {
#pragma unroll
    for (int bp = 0; bp < NB / 2; ++bp)
#pragma unroll
      for (int nb = 0; nb < HDIM / 16; ++nb) {
        const uint2 v0 = v_operand_tr_at<HDIM>(vbase, 2 * bp, nb, lane);
        const uint2 v1 = v_operand_tr_at<HDIM>(vbase, 2 * bp + 1, nb, lane);
        const uint4 vb = make_uint4(v0.x, v0.y, v1.x, v1.y);
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k32(pf.w[bp][rr], vb, st.o[rr][nb]);
      }
  } else {
#pragma unroll
    for (int bi = 0; bi < NB; ++bi)
#pragma unroll
      for (int nb = 0; nb < HDIM / 16; ++nb) {
        const uint2 vb = v_operand_tr_at<HDIM>(vbase, bi, nb, lane);
#pragma unroll
        for (int rr = 0; rr < RPW; ++rr) st.o[rr][nb] = mfma_k16(pf.h[bi][rr], vb, st.o[rr][nb]);
      }
  }
}

}  // namespace hs2
