// Chunked-prefill attention over a mixed-fidelity paged prefix for gfx950
// (paper §3.2: BASE blocks are read as their high bytes with a zero low
// byte; App. A: a prefill chunk attends its cached prefix and, causally,
// itself).
//
// A workgroup of 4 waves serves one (sequence, KV head, tile of query
// tokens).  Its query "columns" are (token, head-in-group) pairs, 16 per
// MFMA column group; each wave owns NCG groups, so one K/V block brought
// into LDS feeds 4 * 16 * NCG query columns.  K/V blocks stream through an
// LDS ring shared by the four waves (each wave issues a quarter of every
// slot's direct-to-LDS loads, then the waves meet at a barrier); a slot is
// one TARGET block or one packed BASE pair, exactly as in decode, and the
// per-slot math (QK^T on 16x16x32 MFMA, online softmax, PV with P split into
// a 16-bit head and remainder) is the decode's.  Column c of group q sees
// kv tokens p < lim(c) = prefix + (its chunk index) + 1.
//
// Block-table entries and tags are fetched per window of 64 blocks; the
// ring drains at window boundaries.
#include "attn_device.h"

namespace ekv {
namespace {

constexpr int kPrefillWaves = 4;
constexpr int kPrefillSlots = 3;
constexpr int kPrefillWindow = 64;

__device__ __forceinline__ void barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <typename T, int G, bool ELASTIC, int NCG>
__global__ __launch_bounds__(256) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) char ring[kPrefillSlots][kSlotBytes];
  constexpr int kTokPerGroup = 16 / G;
  constexpr int kTileTok = kPrefillWaves * NCG * kTokPerGroup;
  const int s = blockIdx.z;
  const int kvh = blockIdx.y;
  const int tile = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int n = lane & 15;
  const int g = lane >> 4;
  const int q0 = a.cu_q[s];
  const int nq = a.cu_q[s + 1] - q0;
  const int t_begin = tile * kTileTok;
  if (t_begin >= nq) return;   // uniform over the workgroup
  const int len = max(0, min(a.seq_lens[s], a.max_blocks * kPage));
  const int prefix = len - nq;

  // this wave's query columns
  u32x4 qop[NCG][4];
  int lim[NCG], lim_min[NCG], tq[NCG];
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    const int t_first = t_begin + (wave * NCG + cg) * kTokPerGroup;
    tq[cg] = t_first + n / G;
    const int h = n % G;
    const bool ok = tq[cg] < nq;
    lim[cg] = ok ? min(len, prefix + tq[cg] + 1) : len;
    lim_min[cg] = min(len, prefix + t_first + 1);
    const uint16_t* qrow = a.q + ((size_t)(q0 + (ok ? tq[cg] : 0)) * a.num_q_heads + (size_t)kvh * G + h) * kHeadDim;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      qop[cg][k] = ok ? *reinterpret_cast<const u32x4*>(qrow + 8 * (4 * g + k)) : u32x4{0u, 0u, 0u, 0u};
  }
  const int t_last = min(nq, t_begin + kTileTok) - 1;
  const int kv_end = max(1, min(len, prefix + t_last + 1));
  const int nblk = (kv_end + kPage - 1) / kPage;

  // mode of the sequence
  int base_lo = 0, base_hi = 0;
  bool use_tags = false;
  if constexpr (ELASTIC) {
    int b0 = -1, b1 = -1;
    if (a.bounds) {
      b0 = a.bounds[2 * s];
      b1 = a.bounds[2 * s + 1];
    }
    if (b0 >= 0) {
      base_lo = 2 * b0;
      base_hi = 2 * b1;
    } else if (a.tags) {
      use_tags = true;
    }
  }

  uint32_t rk_t[4], rv_t[4], rk_b[2], rv_b[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) rk_t[k] = n * (2 * kHeadDim) + 16 * ((4 * g + k) ^ n);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = 4 * g + i;
    rv_t[i] = kTileBytes + t * (2 * kHeadDim) + 16 * (n ^ t);
    rv_b[i] = kTileBytes + t * kHeadDim + 16 * ((n >> 1) ^ tau(t)) + 8 * (n & 1);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) rk_b[h] = n * kHeadDim + 16 * ((2 * g + h) ^ tau(n));
  // each wave loads quarter `wave` of every 4 KiB plane tile of a slot
  const DmaOffsets dma = dma_offsets(lane + 64 * wave);   // row `wave` of the per-lane offsets
  const size_t block_bytes = (size_t)2 * a.num_kv_heads * kTileBytes;
  const char* pool = reinterpret_cast<const char*>(a.pool) + (size_t)kvh * kTileBytes;
  const size_t v_off = (size_t)a.num_kv_heads * kTileBytes;
  const int32_t* btrow = a.bt + (size_t)s * a.max_blocks;

  SplitState st[NCG];
#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
#pragma unroll
    for (int j = 0; j < 8; ++j) st[cg].o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[cg].m = -__builtin_inff();
    st[cg].l = 0.f;
  }

  for (int w0 = 0; w0 < nblk; w0 += kPrefillWindow) {
    const int w1 = min(nblk, w0 + kPrefillWindow);
    const int nw = w1 - w0;
    int bt_lane = lane < nw ? btrow[w0 + lane] : 0;
    bt_lane = (unsigned)bt_lane < (unsigned)a.num_blocks ? bt_lane : 0;   // never leave the pool
    const int tag_lane = (use_tags && lane < nw) ? a.tags[(size_t)s * a.max_blocks + w0 + lane] : 0;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    auto is_base = [&](int blk) -> bool {
      if constexpr (!ELASTIC) return false;
      else return use_tags ? (__builtin_amdgcn_readlane(tag_lane, blk - w0) != 0)
                           : (blk >= base_lo && blk < base_hi);
    };
    int ib = w0, cb = w0, issued = 0, consumed = 0, islot = 0, cslot = 0;
    auto issue = [&]() {
      const bool base = is_base(ib);
      const char* src = pool + (size_t)__builtin_amdgcn_readlane(bt_lane, ib - w0) * block_bytes;
      char* dst = ring[islot];
      const uint32_t off = base ? dma.base[0] : dma.tgt[0];
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + off), (lds_ptr)(dst + 1024 * wave), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + v_off + off),
                                       (lds_ptr)(dst + kTileBytes + 1024 * wave), 16, 0, 0);
      ib += base ? 2 : 1;
      ++issued;
      islot = islot + 1 == kPrefillSlots ? 0 : islot + 1;
    };
#pragma unroll
    for (int k = 0; k < kPrefillSlots - 1; ++k)
      if (ib < w1) issue();
    while (cb < w1) {
      const int ahead = issued - consumed - 1;
      if (ahead >= 2) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
      else if (ahead == 1) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
      else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      barrier();   // every wave's quarter of this slot has landed; the slot reused next is free
      if (ib < w1) issue();
      const char* sb = ring[cslot];
      const int tok0 = cb * kPage;
      if (is_base(cb)) {
        u32x4 k[2][4], v[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const char* mb = sb + m * (kTileBytes / 2);
          const u32x4 k0 = *reinterpret_cast<const u32x4*>(mb + rk_b[0]);
          const u32x4 k1 = *reinterpret_cast<const u32x4*>(mb + rk_b[1]);
          k[m][0].xy = k0.xy;
          k[m][1].xy = k0.zw;
          k[m][2].xy = k1.xy;
          k[m][3].xy = k1.zw;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[m][i].xy = *reinterpret_cast<const u32x2*>(mb + rv_b[i]);
        }
        u32x2 vop[2][8];
        v_operands<true, 2>(v, vop);
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg) {
          const f32x4 sc[2] = {qk_scores<T, true>(k[0], qop[cg]), qk_scores<T, true>(k[1], qop[cg])};
          softmax_pv<T, 2>(st[cg], sc, vop, tok0, lim[cg], tok0 + 2 * kPage > lim_min[cg], a.scale_log2, g);
        }
        cb += 2;
      } else {
        u32x4 k[4], v[1][4];
#pragma unroll
        for (int q = 0; q < 4; ++q) k[q] = *reinterpret_cast<const u32x4*>(sb + rk_t[q]);
#pragma unroll
        for (int i = 0; i < 4; ++i) v[0][i] = *reinterpret_cast<const u32x4*>(sb + rv_t[i]);
        zero_tail_v<1>(v, tok0, len, g);
        u32x2 vop[1][8];
        v_operands<false, 1>(v, vop);
#pragma unroll
        for (int cg = 0; cg < NCG; ++cg) {
          const f32x4 sc[1] = {qk_scores<T, false>(k, qop[cg])};
          softmax_pv<T, 1>(st[cg], sc, vop, tok0, lim[cg], tok0 + kPage > lim_min[cg], a.scale_log2, g);
        }
        cb += 1;
      }
      ++consumed;
      cslot = cslot + 1 == kPrefillSlots ? 0 : cslot + 1;
    }
    barrier();   // the ring is reused by the next window
  }

#pragma unroll
  for (int cg = 0; cg < NCG; ++cg) {
    const float l = head_sum(st[cg].l);
    if (tq[cg] < nq) {
      const float inv = 1.0f / l;
      const size_t row = ((size_t)(q0 + tq[cg]) * a.num_q_heads + (size_t)kvh * G + n % G) * kHeadDim;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        store_row8<T>(a.out, row + 32 * g + 8 * r,
                      f32x4{st[cg].o[0][r], st[cg].o[1][r], st[cg].o[2][r], st[cg].o[3][r]} * inv,
                      f32x4{st[cg].o[4][r], st[cg].o[5][r], st[cg].o[6][r], st[cg].o[7][r]} * inv, a.out_fp32);
    }
  }
}

template <typename T, int G>
hipError_t launch_typed(const PrefillArgs& a, bool elastic, hipStream_t st) {
  constexpr int kNcg = 2;
  constexpr int kTileTok = kPrefillWaves * kNcg * (16 / G);
  dim3 grid((a.max_q_len + kTileTok - 1) / kTileTok, a.num_kv_heads, a.batch);
  if (elastic) hipLaunchKernelGGL((prefill_kernel<T, G, true, kNcg>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((prefill_kernel<T, G, false, kNcg>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_group(const PrefillArgs& a, int group, bool elastic, hipStream_t st) {
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

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int group, bool elastic, hipStream_t st) {
  if (a.batch == 0 || a.max_q_len == 0) return hipSuccess;
  return dtype == 0 ? launch_group<Bf16>(a, group, elastic, st) : launch_group<Fp16>(a, group, elastic, st);
}

}  // namespace ekv
