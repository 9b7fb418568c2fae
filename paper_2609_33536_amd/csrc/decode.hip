// Dual-mode split-KV decode attention for gfx950 (paper §3.2; App. B.3).
//
// One wave (64 lanes) owns one (sequence, KV head, split) work item and
// streams that split's 16-token KV blocks through the block table.  For
// each block it forms S^T = K Q^T for the whole query group with one
// 16x16x32 MFMA chain (tokens x heads, head dim reduced in 4 steps), runs
// an online softmax, and accumulates O^T += V^T P^T with 16x16x16 MFMAs.
//
// Lane (n, g) = (lane & 15, lane >> 4):
//   QK   A operand: token n of the block, head-dim chunk 4*step + g (8 elems)
//        B operand: query head n of the group, same chunk (zero if n >= G)
//        result:    scores of head n for tokens 4g .. 4g+3
//   PV   A operand: V[4g+i][8n + j] for i = 0..3 (MFMA j = 0..7)
//        B operand: the lane's own 4 probabilities (no shuffle needed)
//        result:    O[head n][d], d = 32g + 8r + j, r = 0..3
// so each lane loads 4 x 16 B of K and 4 x 16 B of V per TARGET block (half
// that per BASE block), every load instruction of the wave reading whole
// 256 B token rows (V) or 64 B row segments (K).
//
// TARGET blocks are used as stored.  BASE blocks are read from the packed
// pair block (member i & 1) and widened in registers: byte -> high byte of
// the 16-bit word, zero low byte; one v_perm_b32 per two elements.
//
// The native instantiation never reads tags.  The elastic one decides each
// block's mode from the sequence's boundaries (structured) or from its tag
// row (general); both are wave-uniform scalar branches.
//
// P is split into a 16-bit head and a 16-bit remainder and both are
// multiplied with V, so the PV product carries ~16 significant bits of P.
#include "common.h"
#include "launch.h"

namespace ekv {
namespace {

struct Tile {
  u32x4 k[4];   // TARGET: 4 x 8 words; BASE: .xy = 8 bytes
  u32x4 v[4];
};

template <bool BASE>
__device__ __forceinline__ void load_tile(Tile& t, const uint16_t* ktile, const uint16_t* vtile,
                                          int member, int n, int g) {
  if constexpr (BASE) {
    const uint8_t* kb = reinterpret_cast<const uint8_t*>(ktile) + member * (kTileBytes / 2);
    const uint8_t* vb = reinterpret_cast<const uint8_t*>(vtile) + member * (kTileBytes / 2);
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x2 x = *reinterpret_cast<const u32x2*>(kb + n * kHeadDim + 8 * (4 * st + g));
      t.k[st] = u32x4{x.x, x.y, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      u32x2 x = *reinterpret_cast<const u32x2*>(vb + (4 * g + i) * kHeadDim + 8 * n);
      t.v[i] = u32x4{x.x, x.y, 0u, 0u};
    }
  } else {
#pragma unroll
    for (int st = 0; st < 4; ++st)
      t.k[st] = *reinterpret_cast<const u32x4*>(ktile + n * kHeadDim + 8 * (4 * st + g));
#pragma unroll
    for (int i = 0; i < 4; ++i)
      t.v[i] = *reinterpret_cast<const u32x4*>(vtile + (4 * g + i) * kHeadDim + 8 * n);
  }
}

template <typename T>
struct SplitState {
  f32x4 o[8];
  float m;   // running max, log2 units (same in the 4 lanes of a head)
  float l;   // running sum, partial per lane
};

template <typename T, bool BASE>
__device__ __forceinline__ void consume_tile(SplitState<T>& st, Tile& t, const u32x4 (&qop)[4],
                                             int tok0, int len, float scale_log2) {
  // scores S^T[token][head]
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    u32x4 kop;
    if constexpr (BASE) kop = expand_base8(u32x2{t.k[k].x, t.k[k].y});
    else kop = t.k[k];
    s = Mma<T>::qk(kop, qop[k], s);
  }
  float sc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) sc[i] = (tok0 + i < len) ? s[i] * scale_log2 : -__builtin_inff();
  float mx = fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(st.m, mx);
  const float alpha = fast_exp2(st.m - m_new);
  float p[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = fast_exp2(sc[i] - m_new);
  st.l = st.l * alpha + ((p[0] + p[1]) + (p[2] + p[3]));
  st.m = m_new;
#pragma unroll
  for (int j = 0; j < 8; ++j) st.o[j] *= alpha;

  // P = head + remainder, both as 16-bit operands
  uint16_t ph[4], pl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float back, dummy;
    ph[i] = Mma<T>::round(p[i], &back);
    pl[i] = Mma<T>::round(p[i] - back, &dummy);
  }
  const u32x2 phi = {(uint32_t)ph[0] | ((uint32_t)ph[1] << 16), (uint32_t)ph[2] | ((uint32_t)ph[3] << 16)};
  const u32x2 plo = {(uint32_t)pl[0] | ((uint32_t)pl[1] << 16), (uint32_t)pl[2] | ((uint32_t)pl[3] << 16)};

  // tokens past the end of the sequence may hold anything: zero their V
  if (len - (tok0 & ~15) < kPage) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (tok0 + i >= len) t.v[i] = u32x4{0u, 0u, 0u, 0u};
  }

#pragma unroll
  for (int j = 0; j < 8; ++j) {
    u32x2 vop;
    if constexpr (BASE) {
      // byte j of the lane's 8-byte row segment, for tokens 4g .. 4g+3
      const int b = j & 3;
      const uint32_t sel = 0x0Cu | ((uint32_t)b << 8) | (0x0Cu << 16) | ((uint32_t)(4 + b) << 24);
      const uint32_t w0 = (j < 4) ? t.v[0].x : t.v[0].y;
      const uint32_t w1 = (j < 4) ? t.v[1].x : t.v[1].y;
      const uint32_t w2 = (j < 4) ? t.v[2].x : t.v[2].y;
      const uint32_t w3 = (j < 4) ? t.v[3].x : t.v[3].y;
      vop = u32x2{perm(w1, w0, sel), perm(w3, w2, sel)};
    } else {
      // 16-bit element j of the lane's 8-element row segment
      const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
      vop = u32x2{perm(t.v[1][j >> 1], t.v[0][j >> 1], sel), perm(t.v[3][j >> 1], t.v[2][j >> 1], sel)};
    }
    st.o[j] = Mma<T>::pv(vop, phi, st.o[j]);
    st.o[j] = Mma<T>::pv(vop, plo, st.o[j]);
  }
}

template <typename T, int G, bool ELASTIC>
__global__ __launch_bounds__(64) void decode_split_kernel(DecodeArgs a) {
  const int s = blockIdx.z;
  const int kvh = blockIdx.y;
  const int split = blockIdx.x;
  const int len = a.seq_lens[s];
  const int nblk = (len + kPage - 1) / kPage;
  const int b_begin = split * a.split_blocks;
  if (b_begin >= nblk) return;
  const int b_end = min(nblk, b_begin + a.split_blocks);
  const int nsplit = (nblk + a.split_blocks - 1) / a.split_blocks;

  const int lane = threadIdx.x;
  const int n = lane & 15;
  const int g = lane >> 4;
  const int hkv = a.num_kv_heads;
  const size_t block_words = (size_t)2 * hkv * kTileWords;
  const uint16_t* pool_k = a.pool + (size_t)kvh * kTileWords;
  const size_t v_off = (size_t)hkv * kTileWords;
  const int32_t* btrow = a.bt + (size_t)s * a.max_blocks;

  u32x4 qop[4];
  {
    const uint16_t* qrow = a.q + ((size_t)s * a.num_q_heads + (size_t)kvh * G + n) * kHeadDim;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      qop[k] = (n < G) ? *reinterpret_cast<const u32x4*>(qrow + 8 * (4 * k + g)) : u32x4{0u, 0u, 0u, 0u};
  }

  // per-sequence mode description (wave-uniform)
  int base_lo = 0, base_hi = 0;
  const uint8_t* tagrow = nullptr;
  if constexpr (ELASTIC) {
    int b0 = -1, b1 = -1;
    if (a.bounds) {
      b0 = a.bounds[2 * s];
      b1 = a.bounds[2 * s + 1];
    }
    if (b0 >= 0) {
      base_lo = 2 * b0;
      base_hi = 2 * b1;
    } else {
      tagrow = a.tags + (size_t)s * a.max_blocks;
    }
  }
  auto is_base = [&](int blk) -> bool {
    if constexpr (!ELASTIC) return false;
    else return tagrow ? (tagrow[blk] != 0) : (blk >= base_lo && blk < base_hi);
  };
  auto issue = [&](Tile& t, int blk, bool base) {
    const uint16_t* kt = pool_k + (size_t)btrow[blk] * block_words;
    if (base) load_tile<true>(t, kt, kt + v_off, blk & 1, n, g);
    else load_tile<false>(t, kt, kt + v_off, blk & 1, n, g);
  };

  SplitState<T> st;
#pragma unroll
  for (int j = 0; j < 8; ++j) st.o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -__builtin_inff();
  st.l = 0.f;

  // software pipeline: the next block's loads are in flight while this one
  // is consumed (two register buffers, unrolled by two)
  Tile ta, tb;
  bool base_a = is_base(b_begin), base_b = false;
  issue(ta, b_begin, base_a);
  for (int blk = b_begin; blk < b_end; blk += 2) {
    const bool has_b = blk + 1 < b_end;
    if (has_b) {
      base_b = is_base(blk + 1);
      issue(tb, blk + 1, base_b);
    }
    if (base_a) consume_tile<T, true>(st, ta, qop, blk * kPage + 4 * g, len, a.scale_log2);
    else consume_tile<T, false>(st, ta, qop, blk * kPage + 4 * g, len, a.scale_log2);
    if (!has_b) break;
    const bool has_a = blk + 2 < b_end;
    if (has_a) {
      base_a = is_base(blk + 2);
      issue(ta, blk + 2, base_a);
    }
    if (base_b) consume_tile<T, true>(st, tb, qop, (blk + 1) * kPage + 4 * g, len, a.scale_log2);
    else consume_tile<T, false>(st, tb, qop, (blk + 1) * kPage + 4 * g, len, a.scale_log2);
  }

  float l = st.l;
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  if (n >= G) return;
  const size_t head = (size_t)s * a.num_q_heads + (size_t)kvh * G + n;
  if (nsplit == 1) {
    const float inv = 1.0f / l;
    if (a.out_fp32) {
      float* dst = reinterpret_cast<float*>(a.out) + head * kHeadDim + 32 * g;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        *reinterpret_cast<f32x4*>(dst + 8 * r) =
            f32x4{st.o[0][r], st.o[1][r], st.o[2][r], st.o[3][r]} * inv;
        *reinterpret_cast<f32x4*>(dst + 8 * r + 4) =
            f32x4{st.o[4][r], st.o[5][r], st.o[6][r], st.o[7][r]} * inv;
      }
    } else {
      uint16_t* dst = reinterpret_cast<uint16_t*>(a.out) + head * kHeadDim + 32 * g;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
          float b;
          w[j >> 1] = (uint32_t)Mma<T>::round(st.o[j][r] * inv, &b) |
                      ((uint32_t)Mma<T>::round(st.o[j + 1][r] * inv, &b) << 16);
        }
        *reinterpret_cast<u32x4*>(dst + 8 * r) = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
    return;
  }
  const size_t slot = head * a.max_splits + split;
  float* dst = a.ws_o + slot * kHeadDim + 32 * g;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    *reinterpret_cast<f32x4*>(dst + 8 * r) = f32x4{st.o[0][r], st.o[1][r], st.o[2][r], st.o[3][r]};
    *reinterpret_cast<f32x4*>(dst + 8 * r + 4) = f32x4{st.o[4][r], st.o[5][r], st.o[6][r], st.o[7][r]};
  }
  if (g == 0) *reinterpret_cast<float2*>(a.ws_ml + 2 * slot) = make_float2(st.m, l);
}

// Merge the splits of one (sequence, query head): weights exp2(m_k - M).
template <typename T>
__global__ __launch_bounds__(kHeadDim) void decode_reduce_kernel(DecodeArgs a) {
  const int h = blockIdx.x;
  const int s = blockIdx.y;
  const int d = threadIdx.x;
  const int len = a.seq_lens[s];
  const int nblk = (len + kPage - 1) / kPage;
  const int nsplit = (nblk + a.split_blocks - 1) / a.split_blocks;
  if (nsplit == 1) return;   // the split kernel wrote the final row
  const size_t head = (size_t)s * a.num_q_heads + h;
  float res = 0.f;
  if (nsplit > 1) {
    const float* ml = a.ws_ml + 2 * head * a.max_splits;
    float mmax = -__builtin_inff();
    for (int k = 0; k < nsplit; ++k) mmax = fmaxf(mmax, ml[2 * k]);
    float num = 0.f, den = 0.f;
    const float* o = a.ws_o + head * a.max_splits * kHeadDim + d;
    for (int k = 0; k < nsplit; ++k) {
      const float w = fast_exp2(ml[2 * k] - mmax);
      den += w * ml[2 * k + 1];
      num += w * o[(size_t)k * kHeadDim];
    }
    res = num / den;
  }
  if (a.out_fp32) {
    reinterpret_cast<float*>(a.out)[head * kHeadDim + d] = res;
  } else {
    float b;
    reinterpret_cast<uint16_t*>(a.out)[head * kHeadDim + d] = Mma<T>::round(res, &b);
  }
}

template <typename T, int G>
hipError_t launch_typed(const DecodeArgs& a, bool elastic, hipStream_t st) {
  dim3 grid(a.max_splits, a.num_kv_heads, a.batch);
  if (elastic) hipLaunchKernelGGL((decode_split_kernel<T, G, true>), grid, dim3(64), 0, st, a);
  else hipLaunchKernelGGL((decode_split_kernel<T, G, false>), grid, dim3(64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_reduce_kernel<T>), dim3(a.num_q_heads, a.batch), dim3(kHeadDim), 0, st, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_group(const DecodeArgs& a, int group, bool elastic, hipStream_t st) {
  switch (group) {
    case 1: return launch_typed<T, 1>(a, elastic, st);
    case 2: return launch_typed<T, 2>(a, elastic, st);
    case 4: return launch_typed<T, 4>(a, elastic, st);
    case 8: return launch_typed<T, 8>(a, elastic, st);
    case 16: return launch_typed<T, 16>(a, elastic, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int dtype, int group, bool elastic, hipStream_t st) {
  if (a.batch == 0) return hipSuccess;
  return dtype == 0 ? launch_group<Bf16>(a, group, elastic, st) : launch_group<Fp16>(a, group, elastic, st);
}

}  // namespace ekv
