// Device building blocks shared by the decode and prefill attention kernels
// (internal header): the LDS slot layout and its XOR swizzle, direct-to-LDS
// tile loads, the QK^T / online-softmax / PV steps on MFMA, and output
// stores.  See decode.hip for the lane layout of the matrix operands.
#pragma once

#include "common.h"
#include "launch.h"

namespace ekv {
namespace {

constexpr int kSlotBytes = 2 * kTileBytes;   // K tile + V tile

// XOR swizzle of 16-byte chunks inside an LDS tile.
//  TARGET tile: 16 token rows x 16 chunks; chunk c of token t sits at c ^ t.
//  BASE tile: 2 members x 16 rows x 8 chunks; chunk q of token t at q ^ tau(t).
__device__ __forceinline__ int tau(int t) { return (t & 7) ^ (t >> 3); }

// Byte offsets, within a 4 KiB plane tile in HBM, of the 16 B each lane
// fetches with load instruction r (LDS destination: r * 1 KiB + 16 * lane).
struct DmaOffsets {
  uint32_t tgt[4], base[4];
};

__device__ __forceinline__ DmaOffsets dma_offsets(int lane) {
  DmaOffsets o;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int p = 64 * r + lane;                 // LDS chunk written by this lane
    const int t = p >> 4, pos = p & 15;
    o.tgt[r] = t * (2 * kHeadDim) + 16 * (pos ^ t);
    const int m = p >> 7, tb = (p >> 3) & 15, posb = p & 7;
    o.base[r] = m * (kTileBytes / 2) + tb * kHeadDim + 16 * (posb ^ tau(tb));
  }
  return o;
}

typedef __attribute__((address_space(3))) void* lds_ptr;

// Cache policy of the K/V tile loads of decode: non-temporal.  Decode reads
// every K/V byte of a launch exactly once, so keeping the lines in the
// caches only displaces other data; with the non-temporal bit the
// direct-to-LDS stream of random 8 KiB tiles reads 6.9 TB/s on MI355X,
// against 6.2 TB/s with the default policy.  (Prefill re-reads each tile
// for every query tile of its sequence and keeps the default.)
constexpr int kStreamOnce = 2;   // the NT bit of the load's cache-policy operand

// A lane's 32-bit offset, made opaque at the load: without it the compiler
// hoists the offset's widening to 64 bits out of the loop, and each load then
// needs a 64-bit vector add for its address; with it the load takes the
// scalar-base form (64-bit base in scalar registers + 32-bit lane offset).
__device__ __forceinline__ uint32_t lane_offset(uint32_t off) {
  asm volatile("" : "+v"(off));
  return off;
}

__device__ __forceinline__ void dma_tile(const char* src, const uint32_t (&off)[4], char* dst) {
#pragma unroll
  for (int r = 0; r < 4; ++r)
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + lane_offset(off[r])),
                                     (lds_ptr)(dst + 1024 * r), 16, 0, kStreamOnce);
}

struct SplitState {
  f32x4 o[8];
  float m;   // reference max, log2 units (same in the 4 lanes of a head)
  float l;   // running sum, partial per lane
};

// max / sum over the four lanes of one head (lanes l, l^16, l^32, l^48)
__device__ __forceinline__ float head_max(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float head_sum(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// PV A operand for MFMA j (head-dim row 8n + j): the lane's 4 tokens, as
// 16-bit words.  TARGET rows hold 8 words per token, BASE rows 8 bytes.
template <bool BASE>
__device__ __forceinline__ u32x2 v_operand(const u32x4 (&v)[4], int j) {
  if constexpr (BASE) {
    const int b = j & 3;
    const uint32_t sel = 0x0Cu | ((uint32_t)b << 8) | (0x0Cu << 16) | ((uint32_t)(4 + b) << 24);
    const int w = j >> 2;
    return u32x2{perm(v[1][w], v[0][w], sel), perm(v[3][w], v[2][w], sel)};
  } else {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
    return u32x2{perm(v[1][j >> 1], v[0][j >> 1], sel), perm(v[3][j >> 1], v[2][j >> 1], sel)};
  }
}

// Scores of one 16-token group: S^T = K Q^T, lane gets tokens 4g..4g+3 of head n.
template <typename T, bool BASE>
__device__ __forceinline__ f32x4 qk_scores(const u32x4 (&k)[4], const u32x4 (&qop)[4]) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    u32x4 kop;
    if constexpr (BASE) kop = expand_base8(k[st].xy);
    else kop = k[st];
    s = Mma<T>::qk(kop, qop[st], s);
  }
  return s;
}

// Zero the V rows of tokens at or past the sequence end (their slots may
// hold anything, and 0 * NaN would poison the product).
template <int NG>
__device__ __forceinline__ void zero_tail_v(u32x4 (&v)[NG][4], int tok0, int len, int g) {
  if (tok0 + NG * kPage > len) {
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (tok0 + q * kPage + 4 * g + i >= len) v[q][i] = u32x4{0u, 0u, 0u, 0u};
  }
}

template <bool BASE, int NG>
__device__ __forceinline__ void v_operands(const u32x4 (&v)[NG][4], u32x2 (&vop)[NG][8]) {
#pragma unroll
  for (int q = 0; q < NG; ++q)
#pragma unroll
    for (int j = 0; j < 8; ++j) vop[q][j] = v_operand<BASE>(v[q], j);
}

// The A operands of the column-stacked PV product: operand j holds the
// lane's 4 tokens of group 0 and then those of group 1 (zero for NG = 1),
// built in place, so that no register moves sit between the permutes and
// the products.
template <bool BASE, int NG>
__device__ __forceinline__ void v_operands_stacked(const u32x4 (&v)[NG][4], u32x4 (&vop)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const u32x2 a0 = v_operand<BASE>(v[0], j);
    const u32x2 a1 = NG == 2 ? v_operand<BASE>(v[NG - 1], j) : u32x2{0u, 0u};
    vop[j] = u32x4{a0.x, a0.y, a1.x, a1.y};
  }
}

// Two probabilities -> one packed word for the column-stacked product: the
// 16-bit heads rne(p) for k = 0 (head columns), the 16-bit remainders
// rne(p - rne(p)) for k = 1 (remainder columns).  p - rne(p) is exact in
// fp32, so one fused multiply-add per value selects what is rounded.
template <typename T>
__device__ __forceinline__ uint32_t split_stacked(float p0, float p1, float k);
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float f32x2v __attribute__((ext_vector_type(2)));
template <>
__device__ __forceinline__ uint32_t split_stacked<Bf16>(float p0, float p1, float k) {
  const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2v{p0, p1}, bf16x2v));
  const f32x2v v = {__builtin_fmaf(-k, __uint_as_float(h << 16), p0),
                    __builtin_fmaf(-k, __uint_as_float(h & 0xffff0000u), p1)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2v));
}
template <>
__device__ __forceinline__ uint32_t split_stacked<Fp16>(float p0, float p1, float k) {
  const _Float16 h0 = (_Float16)p0, h1 = (_Float16)p1;
  const _Float16 w0 = (_Float16)__builtin_fmaf(-k, (float)h0, p0), w1 = (_Float16)__builtin_fmaf(-k, (float)h1, p1);
  return (uint32_t)__builtin_bit_cast(uint16_t, w0) | ((uint32_t)__builtin_bit_cast(uint16_t, w1) << 16);
}

// Online-softmax update of one query column set for NG 16-token groups of
// one slot, followed by O += V^T P^T.  c = |scale| log2(e) >= 0: a negative
// scale is applied by negating the query (exact) instead.  Token p of group q (p = tok0 + 16q
// + 4g + i for this lane) counts only if p < lim (lim: this lane's column
// limit); `mask` says whether any token of the slot can fail that test.
// The reference max only moves (and O, l are rescaled) when some column's
// block max exceeds it by more than 2^8; otherwise P <= 2^8.  P is split
// into a 16-bit head and remainder, stacked along k of one 16x16x32 MFMA
// against the duplicated V operand.
template <typename T, int NG>
__device__ __forceinline__ void softmax_pv(SplitState& st, const f32x4 (&s)[NG], const u32x2 (&vop)[NG][8],
                                           int tok0, int lim, bool mask, float c, int g) {
  float sc[NG][4];
#pragma unroll
  for (int q = 0; q < NG; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) sc[q][i] = s[q][i] * c;
  if (mask) {
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (tok0 + q * kPage + 4 * g + i >= lim) sc[q][i] = -__builtin_inff();
  }
  float mx = fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3]));
#pragma unroll
  for (int q = 1; q < NG; ++q) mx = fmaxf(mx, fmaxf(fmaxf(sc[q][0], sc[q][1]), fmaxf(sc[q][2], sc[q][3])));
  mx = head_max(mx);
  if (__builtin_amdgcn_ballot_w64(mx > st.m + 8.0f)) {
    const float m_new = fmaxf(st.m, mx);
    const float alpha = fast_exp2(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int j = 0; j < 8; ++j) st.o[j] *= alpha;
    st.m = m_new;
  }
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = fast_exp2(sc[q][i] - st.m);
    st.l += (p[0] + p[1]) + (p[2] + p[3]);
    uint16_t ph[4], pl[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float back, dummy;
      ph[i] = Mma<T>::round(p[i], &back);
      pl[i] = Mma<T>::round(p[i] - back, &dummy);
    }
    const u32x4 pb = {(uint32_t)ph[0] | ((uint32_t)ph[1] << 16), (uint32_t)ph[2] | ((uint32_t)ph[3] << 16),
                      (uint32_t)pl[0] | ((uint32_t)pl[1] << 16), (uint32_t)pl[2] | ((uint32_t)pl[3] << 16)};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const u32x2 a = vop[q][j];
      st.o[j] = Mma<T>::qk(u32x4{a.x, a.y, a.x, a.y}, pb, st.o[j]);
    }
  }
}

// Column-stacked variant for query groups of at most 8 heads: query column
// n < G and column n + G both hold head n (their scores, max and sum agree),
// and one 16x16x32 MFMA per head-dim row set covers 32 tokens (NG = 2: the
// lane's 4 tokens of each of two 16-token groups; NG = 1: one group, the
// other half zero).  Columns n < G accumulate V^T times the 16-bit head of P,
// columns G <= n < 2G the 16-bit remainder; stacked_sum() adds the two
// column sets at the end.  So P still carries ~16 significant bits, and V
// is neither duplicated nor multiplied twice.  Scores enter the softmax as
// s * c (log2 units, c >= 0): a step without masked tokens folds c into the
// max and the exponent's fused multiply-add; a masked step scales first and
// then sets masked tokens to -inf, so that c = 0 never multiplies an infinity.
template <typename T, int NG, int G>
__device__ __forceinline__ void softmax_pv_stacked(SplitState& st, const f32x4 (&s)[NG], const u32x4 (&vop)[8],
                                                   int tok0, int lim, bool mask, float c, int g, int n) {
  static_assert(2 * G <= 16, "two column sets must fit the 16 MFMA columns");
  float sc[NG][4];
  float cc = c;
  if (mask) {
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[q][i] = tok0 + q * kPage + 4 * g + i >= lim ? -__builtin_inff() : s[q][i] * c;
    cc = 1.0f;
  } else {
#pragma unroll
    for (int q = 0; q < NG; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i) sc[q][i] = s[q][i];
  }
  float mx = fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3]));
#pragma unroll
  for (int q = 1; q < NG; ++q) mx = fmaxf(mx, fmaxf(fmaxf(sc[q][0], sc[q][1]), fmaxf(sc[q][2], sc[q][3])));
  mx = head_max(mx) * cc;
  if (__builtin_amdgcn_ballot_w64(mx > st.m + 8.0f)) {
    const float m_new = fmaxf(st.m, mx);
    const float alpha = fast_exp2(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int j = 0; j < 8; ++j) st.o[j] *= alpha;
    st.m = m_new;
  }
  const float k = n >= G ? 1.0f : 0.0f;   // remainder columns
  uint32_t pw[2][2] = {{0u, 0u}, {0u, 0u}};
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = fast_exp2(__builtin_fmaf(sc[q][i], cc, -st.m));
    st.l += (p[0] + p[1]) + (p[2] + p[3]);
    pw[q][0] = split_stacked<T>(p[0], p[1], k);
    pw[q][1] = split_stacked<T>(p[2], p[3], k);
  }
  const u32x4 pb = {pw[0][0], pw[0][1], pw[1][0], pw[1][1]};
#pragma unroll
  for (int j = 0; j < 8; ++j) st.o[j] = Mma<T>::qk(vop[j], pb, st.o[j]);
}

// PV operands of one 32-token step: column-stacked (S, groups of at most 8
// heads) or per 16-token group.  One softmax / PV call per step, whatever
// the kind of the step's blocks, keeps the accumulators in one place: with
// a call per kind, the compiler gave each its own output registers and
// copied all 32 accumulator registers back at the top of every step.
template <bool S>
struct PvOps {
  u32x4 v[8];
};
template <>
struct PvOps<false> {
  u32x2 v[2][8];
};

// NG = 1: the second group's operands are zero (its tokens are masked).
template <bool BASE, int NG, bool S>
__device__ __forceinline__ void pv_operands(const u32x4 (&v)[NG][4], PvOps<S>& o) {
  if constexpr (S) {
    v_operands_stacked<BASE, NG>(v, o.v);
  } else {
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int j = 0; j < 8; ++j) o.v[q][j] = q < NG ? v_operand<BASE>(v[q < NG ? q : 0], j) : u32x2{0u, 0u};
  }
}

template <typename T, int G, bool S>
__device__ __forceinline__ void pv_step(SplitState& st, const f32x4 (&s)[2], const PvOps<S>& o, int tok0, int lim,
                                        bool mask, float c, int g, int n) {
  if constexpr (S) softmax_pv_stacked<T, 2, G>(st, s, o.v, tok0, lim, mask, c, g, n);
  else softmax_pv<T, 2>(st, s, o.v, tok0, lim, mask, c, g);
}

// After column-stacked accumulation: column n (< G) gets its remainder
// column n + G added (lanes n and n + G of each 16-lane row).
template <int G>
__device__ __forceinline__ void stacked_sum(SplitState& st) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) st.o[j][r] += __shfl_xor(st.o[j][r], G);
}

template <typename T>
__device__ __forceinline__ void store_row8(void* out, size_t idx, f32x4 a, f32x4 b, bool fp32) {
  if (fp32) {
    float* dst = reinterpret_cast<float*>(out) + idx;
    *reinterpret_cast<f32x4*>(dst) = a;
    *reinterpret_cast<f32x4*>(dst + 4) = b;
  } else {
    float x;
    uint32_t w[4];
    w[0] = (uint32_t)Mma<T>::round(a[0], &x) | ((uint32_t)Mma<T>::round(a[1], &x) << 16);
    w[1] = (uint32_t)Mma<T>::round(a[2], &x) | ((uint32_t)Mma<T>::round(a[3], &x) << 16);
    w[2] = (uint32_t)Mma<T>::round(b[0], &x) | ((uint32_t)Mma<T>::round(b[1], &x) << 16);
    w[3] = (uint32_t)Mma<T>::round(b[2], &x) | ((uint32_t)Mma<T>::round(b[3], &x) << 16);
    *reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(out) + idx) = u32x4{w[0], w[1], w[2], w[3]};
  }
}

template <typename T>
__device__ __forceinline__ void store_pair(void* out, size_t idx, float a, float b, bool fp32) {
  if (fp32) {
    *reinterpret_cast<float2*>(reinterpret_cast<float*>(out) + idx) = make_float2(a, b);
  } else {
    float x;
    *reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(out) + idx) =
        (uint32_t)Mma<T>::round(a, &x) | ((uint32_t)Mma<T>::round(b, &x) << 16);
  }
}


}  // namespace
}  // namespace ekv
