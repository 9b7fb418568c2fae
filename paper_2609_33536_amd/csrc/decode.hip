// Dual-mode split-KV decode attention for gfx950 (paper §3.2; App. B.3).
//
// One wave (64 lanes) per workgroup.  The work -- every pair of 16-token
// KV blocks of every (sequence, KV head) -- is flattened and cut into equal
// contiguous ranges, one per workgroup of a persistent grid; a wave streams
// its range's blocks through the block table, crossing (sequence, KV head)
// boundaries.  For each block it forms S^T = K Q^T for the whole query
// group with one 16x16x32 MFMA chain (tokens x heads, head dim reduced in 4
// steps), runs an online softmax over 32-token steps, and accumulates
// O^T += V^T P^T with 16x16x16 MFMAs.
//
// Lane (n, g) = (lane & 15, lane >> 4):
//   QK   A operand: token n of the block, head-dim chunk 4*g + step (8 elems)
//        B operand: query head n % G of the group, same chunk (zero for
//        unused columns)
//        result:    scores of column n for tokens 4g .. 4g+3
//   PV   A operand: V[4g+i][8n + j] for i = 0..3 (MFMA j = 0..7)
//        B operand: the lane's own 4 probabilities (no shuffle needed)
//        result:    O[column n][d], d = 32g + 8r + j, r = 0..3
// For G <= 8 column n < G carries P's 16-bit head and column n + G its
// 16-bit remainder for the same head, so one product per 16 tokens covers
// both; the two columns are added when a piece ends.
//
// K/V move HBM -> LDS with direct-to-LDS loads (global_load_lds_dwordx4),
// each instruction one coalesced 1 KiB, into a per-wave ring of NSLOT 8 KiB
// slots.  A slot holds the (K, V) 4 KiB tiles of one physical block for this
// KV head: either one TARGET block or one whole packed BASE pair (the pair
// layout puts both members' bytes in exactly one tile per plane), so every
// slot costs the same 8 load instructions and bytes whatever its mode, and
// NSLOT-1 slots stay in flight while one is consumed.  The lane -> address
// map of the loads stores each 16 B chunk at an XOR-swizzled position so
// the MFMA-layout ds_read_b128 / ds_read_b64 reads below hit distinct banks.
// The compiler does not track LDS written by these loads, so the ring waits
// on the load counter itself (s_waitcnt vmcnt) before reading a slot.
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
//
// Pieces of a (sequence, KV head) cut by range ends write fp32 partials
// (o, max, sum); the wave that finishes last -- found with a per-(sequence,
// KV head) counter in the workspace -- merges them and writes the output,
// then resets the counter to zero for the next call.
#include <algorithm>
#include <atomic>

#include "attn_device.h"
#include "common.h"
#include "launch.h"

#ifdef EKV_TIMELINE
// Instrumented build only (libekv_timeline.so): per-workgroup timestamps of
// the last decode launch -- start, first K/V slot ready, end of the stream,
// end of the merges (100 MHz constant clock) -- and the workgroup's XCD,
// for the per-launch time budget.  Not compiled into libekv.so.
__device__ uint64_t g_timeline[8 * 8192];
extern "C" int ekv_timeline_read(uint64_t* host, int n) {
  return (int)hipMemcpyFromSymbol(host, HIP_SYMBOL(g_timeline), sizeof(uint64_t) * n, 0, hipMemcpyDeviceToHost);
}
extern "C" int ekv_timeline_clear(void) {
  static uint64_t zeros[8 * 8192];
  return (int)hipMemcpyToSymbol(HIP_SYMBOL(g_timeline), zeros, sizeof(zeros), 0, hipMemcpyHostToDevice);
}
#define EKV_TL(...) __VA_ARGS__
#else
#define EKV_TL(...)
#endif

namespace ekv {
namespace {

constexpr int kMaxDevices = 64;

__device__ __forceinline__ void store_agent_f2(float* p, float a, float b) {
  const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float2 load_agent_f2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Workspace slots of partials.  Workgroup w owns slots 2w and 2w + 1: the
// piece of the (sequence, KV head) that contains its first pair goes to 2w,
// the piece of a later (sequence, KV head) that contains its last pair to
// 2w + 1 (the (sequence, KV head)s strictly inside its range are never cut).
// Piece k of a cut (sequence, KV head) was made by workgroup w_first + k, so
// its slot is 2 (w_first + k), plus one for k = 0 when the (sequence, KV
// head) starts inside w_first's range (first_odd).  The merge counter of a
// (sequence, KV head) lives at the slot of its piece 0.  A slot holds G
// partial rows (one per query head of the group) and G (max, sum) pairs.
__device__ __forceinline__ int piece_slot(int w_first, int first_odd, int k) {
  return 2 * (w_first + k) + (k == 0 ? first_odd : 0);
}

// A slot holds a piece's G partial rows as 32 G chunks of 16 bytes.  The
// writing lane (n, g), n < G, holds dims 32 g .. 32 g + 31 of head n; its
// chunk ci (dims 32 g + 4 ci .. + 3) sits at chunk ci * 4 G + n + G g, so
// each of its 8 store instructions covers 4 G consecutive chunks (whole
// 64-byte lines).  Chunk q of a slot: ci = q / 4G, n = q % G, g = (q % 4G) / G.
// The stores and loads carry the agent-scope cache policy (sc1: written
// through to, and read from, the memory side, which every XCD sees), as the
// relaxed agent-scope 8-byte atomics do; 16 bytes a lane and whole lines a
// store instruction, where 8-byte stores with a row-major layout cost a
// 32-byte write request per lane (four times the partial bytes in HBM
// writes, and ~5 % of an f = 1 launch's time).  The workspace is 16-byte
// aligned (checked at the entry point).
__device__ __forceinline__ void store_agent_f4(float* p, f32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ f32x4 load_agent_row4(const float* p) {
  f32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// Completes this wave's loads; the registers are tied to the wait so that no
// use of them is scheduled before it.
__device__ __forceinline__ void wait_rows(f32x4 (&v)[16]) {
  asm volatile("s_waitcnt vmcnt(0)"
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]),
                 "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]), "+v"(v[13]), "+v"(v[14]), "+v"(v[15])
               :
               : "memory");
}

// Merge the nsplit (<= 64) partials of the G heads of one (sequence, KV
// head): out = sum_k w_k o_k / sum_k w_k l_k with w_k = exp2(m_k - max m).
// Lane k holds split k's (max, sum).  The numerators follow the slot
// layout: a load of the wave reads 64 consecutive chunks of one split (or,
// for G = 1, the 32 chunks of two splits), so lane L owns head L % G and the
// chunks L + 64 t.  The (max, sum) loads and the first 16 chunk loads are
// issued together: a merge of up to one batch of splits costs one memory
// round trip.
template <typename T, int G>
__device__ void merge_splits(const DecodeArgs& a, size_t head0, int nsplit, int w_first, int first_odd, int lane) {
  constexpr int kT = G >= 2 ? G / 2 : 1;        // loads per split (G = 1: one load covers two splits)
  constexpr int kSB = G >= 2 ? 16 / kT : 32;    // splits per batch of 16 loads
  float2 mlk[G];
#pragma unroll
  for (int h = 0; h < G; ++h)
    mlk[h] = lane < nsplit ? load_agent_f2(a.ws_ml + 2 * ((size_t)piece_slot(w_first, first_odd, lane) * G + h))
                           : make_float2(-__builtin_inff(), 0.f);
  // split and chunk of load i of the batch at k0
  auto split_of = [&](int k0, int i) { return G >= 2 ? k0 + i / kT : k0 + 2 * i + (lane >> 5); };
  auto chunk_of = [&](int i) { return G >= 2 ? lane + 64 * (i % kT) : (lane & 31); };
  f32x4 v[16];
  auto load_batch = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int k = min(split_of(k0, i), nsplit - 1);   // a split that exists (zeroed below if past the last)
      v[i] = load_agent_row4(a.ws_o + (size_t)piece_slot(w_first, first_odd, k) * G * kHeadDim + 4 * chunk_of(i));
    }
  };
  load_batch(0);
  const int my_h = lane % G;
  float wk[G], my_inv = 0.f;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float mmax = wave_max(mlk[h].x);
    wk[h] = lane < nsplit ? fast_exp2(mlk[h].x - mmax) : 0.f;
    const float inv = 1.0f / wave_sum(wk[h] * mlk[h].y);
    my_inv = h == my_h ? inv : my_inv;
  }
  f32x4 num[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) num[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0;;) {
    wait_rows(v);
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (split_of(k0, i) >= nsplit) v[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (G >= 2) {
#pragma unroll
      for (int sp = 0; sp < kSB; ++sp) {
        const int k = min(k0 + sp, 63);
        float w = 0.f;
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const float wh = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk[h]), k));
          w = h == my_h ? wh : w;
        }
#pragma unroll
        for (int t = 0; t < kT; ++t) num[t] += w * v[sp * kT + t];
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int k = k0 + 2 * i;
        const float w0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk[0]), min(k, 63)));
        const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk[0]), min(k + 1, 63)));
        num[0] += ((lane >> 5) ? w1 : w0) * v[i];
      }
    }
    k0 += kSB;
    if (k0 >= nsplit) break;
    load_batch(k0);
  }
  if constexpr (G == 1) {   // the two halves of the wave summed splits of opposite parity
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(num[0][e]), __float_as_uint(num[0][e]),
                                                       false, false);
      num[0][e] = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    }
  }
  if (G >= 2 || lane < 32) {
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      const int q = chunk_of(t);
      const int ci = q / (4 * G), g = (q % (4 * G)) / G;
      const f32x4 tot = num[t] * my_inv;
      const size_t idx = (head0 + my_h) * kHeadDim + 32 * g + 4 * ci;
      store_pair<T>(a.out, idx, tot[0], tot[1], a.out_fp32);
      store_pair<T>(a.out, idx + 2, tot[2], tot[3], a.out_fp32);
    }
  }
}

// Any number of splits, one head (h of the group) at a time (long sequences only).
template <typename T, int G>
__device__ void merge_head_serial(const DecodeArgs& a, size_t head, int h, int nsplit, int w_first, int first_odd,
                                  int lane) {
  const float* ml = a.ws_ml + 2 * h;
  // dims 2 lane, 2 lane + 1: chunk (c % 8) * 4G + h + G (c / 8) of the slot, c = lane / 2
  const int c = lane >> 1;
  const float* o = a.ws_o + 4 * ((c & 7) * 4 * G + h + G * (c >> 3)) + 2 * (lane & 1);
  float mmax = -__builtin_inff();
  for (int k0 = 0; k0 < nsplit; k0 += 64)
    if (k0 + lane < nsplit) mmax = fmaxf(mmax, load_agent_f2(ml + 2 * (size_t)piece_slot(w_first, first_odd, k0 + lane) * G).x);
  mmax = wave_max(mmax);
  float den = 0.f, num0 = 0.f, num1 = 0.f;
  for (int k0 = 0; k0 < nsplit; k0 += 64) {
    float wk = 0.f;
    if (k0 + lane < nsplit) {
      const float2 mlk = load_agent_f2(ml + 2 * (size_t)piece_slot(w_first, first_odd, k0 + lane) * G);
      wk = fast_exp2(mlk.x - mmax);
      den += wk * mlk.y;
    }
    const int kn = min(64, nsplit - k0);
    for (int k = 0; k < kn; ++k) {
      const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wk), k));
      const float2 v = load_agent_f2(o + (size_t)piece_slot(w_first, first_odd, k0 + k) * G * kHeadDim);
      num0 += w * v.x;
      num1 += w * v.y;
    }
  }
  const float inv = 1.0f / wave_sum(den);
  store_pair<T>(a.out, head * kHeadDim + 2 * lane, num0 * inv, num1 * inv, a.out_fp32);
}

// Wait until at most n load/store instructions of this wave are in flight
// (n rounded down to a multiple of 8 -- waiting longer is always safe).
template <int COMMON>
__device__ __forceinline__ void wait_vm(int n) {
  n = __builtin_amdgcn_readfirstlane(n);   // wave-uniform: scalar branches below
  if (n >= 63) return;
  const int k = n >> 3;
  if (k == COMMON) {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(8 * COMMON) : "memory");
    return;
  }
  switch (k) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(16)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt vmcnt(24)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(32)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt vmcnt(40)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(48)" ::: "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(56)" ::: "memory"); break;
  }
}

// As wait_vm, in steps of 4 (units of the 8-bit format cost 4 loads), as
// one assembly block: the largest level L in {0, 4, ..., 32} with L <= n is
// found by a balanced tree of scalar compares (three or four, at most two
// taken branches) and vmcnt(L) is awaited (never more than n).  Written as
// a C switch over its levels, the compiler's control-flow structurizer made
// it a long run of scalar instructions and taken branches on every step,
// which the 8-bit elastic path (bound by instruction latency) paid for.  n
// is at most 4 (units in the ring - 1) + the window's loads, below 36 for
// rings of up to 4 slots.
__device__ __forceinline__ void wait_vm4(int n) {
  n = __builtin_amdgcn_readfirstlane(n);
  asm volatile(
      "s_cmp_lt_i32 %0, 16\n\t"
      "s_cbranch_scc1 1f\n\t"
      "s_cmp_lt_i32 %0, 24\n\t"
      "s_cbranch_scc1 2f\n\t"
      "s_cmp_lt_i32 %0, 28\n\t"
      "s_cbranch_scc1 3f\n\t"
      "s_cmp_lt_i32 %0, 32\n\t"
      "s_cbranch_scc1 4f\n\t"
      "s_waitcnt vmcnt(32)\n\t"
      "s_branch 9f\n"
      "4:\n\t"
      "s_waitcnt vmcnt(28)\n\t"
      "s_branch 9f\n"
      "3:\n\t"
      "s_waitcnt vmcnt(24)\n\t"
      "s_branch 9f\n"
      "2:\n\t"
      "s_cmp_lt_i32 %0, 20\n\t"
      "s_cbranch_scc1 5f\n\t"
      "s_waitcnt vmcnt(20)\n\t"
      "s_branch 9f\n"
      "5:\n\t"
      "s_waitcnt vmcnt(16)\n\t"
      "s_branch 9f\n"
      "1:\n\t"
      "s_cmp_lt_i32 %0, 8\n\t"
      "s_cbranch_scc1 6f\n\t"
      "s_cmp_lt_i32 %0, 12\n\t"
      "s_cbranch_scc1 7f\n\t"
      "s_waitcnt vmcnt(12)\n\t"
      "s_branch 9f\n"
      "7:\n\t"
      "s_waitcnt vmcnt(8)\n\t"
      "s_branch 9f\n"
      "6:\n\t"
      "s_cmp_lt_i32 %0, 4\n\t"
      "s_cbranch_scc1 8f\n\t"
      "s_waitcnt vmcnt(4)\n\t"
      "s_branch 9f\n"
      "8:\n\t"
      "s_waitcnt vmcnt(0)\n"
      "9:" ::"s"(n)
      : "memory", "scc");
}

// ---- 8-bit TARGET / 4-bit BASE slots -------------------------------------
// The ring is cut into 4 KiB units.  A TARGET pair takes two: its K and its
// V tiles, each laid out exactly as one plane of a 16-bit packed BASE pair
// ([member 0 | member 1] rows of 128 bytes, swizzled as in dma_offsets) and
// read by the same byte path, member m fetched from its own block.  A BASE
// pair takes one: K nibbles at +0 and V nibbles at +2 KiB, expanded to bytes
// in registers.  So the bytes in flight do not shrink when pairs are BASE.

// A BASE pair's packed nibble tile (2 KiB: [member][16 rows][64 bytes]),
// 16-byte chunk c of row t stored at chunk position c ^ ((t >> 2) & 3) so
// that the operand reads below spread over the banks.  nib[r]: the source
// offset lane L fetches with load r (LDS destination 1024 r + 16 L).
__device__ __forceinline__ void dma_nibbles(const char* tile, const uint32_t (&nib)[2], char* dst) {
#pragma unroll
  for (int r = 0; r < 2; ++r)
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(tile + lane_offset(nib[r])), (lds_ptr)(dst + 1024 * r), 16,
                                     0, kStreamOnce);
}

// A TARGET pair's tile: loads 0, 1 (member 0) from tile0, 2, 3 (member 1) from tile1.
__device__ __forceinline__ void dma_pair_bytes(const char* tile0, const char* tile1, const uint32_t (&off)[4],
                                               char* dst) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const char* src = r < 2 ? tile0 + lane_offset(off[r]) : tile1 + lane_offset(off[r] - kTileBytes / 2);
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(src), (lds_ptr)(dst + 1024 * r), 16, 0, kStreamOnce);
  }
}

// The lone last block of a sequence: member 0's rows only.
__device__ __forceinline__ void dma_member0_bytes(const char* tile0, const uint32_t (&off)[4], char* dst) {
#pragma unroll
  for (int r = 0; r < 2; ++r)
    __builtin_amdgcn_global_load_lds(static_cast<const void*>(tile0 + lane_offset(off[r])), (lds_ptr)(dst + 1024 * r), 16,
                                     0, kStreamOnce);
}

// The same 4 bytes of nibbles as two byte planes, each nibble in the high
// half of its byte: byte k of `even` holds element 2k, of `odd` element 2k+1.
struct NibPlanes {
  uint32_t even, odd;
};
__device__ __forceinline__ NibPlanes nib_planes(uint32_t w) { return {(w << 4) & 0xF0F0F0F0u, w & 0xF0F0F0F0u}; }

// Byte selector that places byte k of the second source in the high byte
// of the low half and byte k of the first source in the high byte of the
// high half, with zero low bytes (two executed BASE words).
__device__ __forceinline__ constexpr uint32_t word_pair_sel(int k) {
  return 0x0Cu | ((uint32_t)k << 8) | (0x0Cu << 16) | ((uint32_t)(4 + k) << 24);
}

// 8-bit pools: the QK^T operands of a 16-dim step hold its 8 elements as
// 16-bit word pairs (e_j, e_{j+4}), j = 0..3, for K and Q alike (the dot
// product does not depend on the order, as long as both follow it).  BASE K
// then takes one packed 16-bit shift (and a mask) per word: 8 nibbles ->
// 4 words in 6 instructions, where the (e_2j, e_2j+1) order took 7.
typedef unsigned short u16x2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x4 nib_words_x4(uint32_t w) {
  const u16x2v x = __builtin_bit_cast(u16x2v, w);
  constexpr uint32_t kTop = 0xF000F000u;   // the top nibble of each 16-bit half
  return u32x4{__builtin_bit_cast(uint32_t, (u16x2v)(x << 12)), __builtin_bit_cast(uint32_t, (u16x2v)(x << 8)) & kTop,
               __builtin_bit_cast(uint32_t, (u16x2v)(x << 4)) & kTop, w & kTop};
}
// 8 element bytes (a TARGET row or a lone block's, in the byte layout) ->
// words (b_j << 8, b_{j+4} << 8)
__device__ __forceinline__ u32x4 byte_words_x4(u32x2 b) {
  return u32x4{perm(b.y, b.x, word_pair_sel(0)), perm(b.y, b.x, word_pair_sel(1)), perm(b.y, b.x, word_pair_sel(2)),
               perm(b.y, b.x, word_pair_sel(3))};
}
// Q's words (q_2j, q_2j+1) -> (q_j, q_{j+4})
__device__ __forceinline__ u32x4 q_words_x4(u32x4 w) {
  return u32x4{perm(w[2], w[0], 0x05040100u), perm(w[2], w[0], 0x07060302u), perm(w[3], w[1], 0x05040100u),
               perm(w[3], w[1], 0x07060302u)};
}

// PV A operand j of BASE V straight from the planes of the lane's 4 tokens:
// element j of tokens 0 and 1, then of tokens 2 and 3, as 16-bit words.
__device__ __forceinline__ u32x2 nib_v_operand(const NibPlanes (&p)[4], int j) {
  const uint32_t sel = word_pair_sel(j >> 1);
  if (j & 1) return u32x2{perm(p[1].odd, p[0].odd, sel), perm(p[3].odd, p[2].odd, sel)};
  return u32x2{perm(p[1].even, p[0].even, sel), perm(p[3].even, p[2].even, sel)};
}

__device__ __forceinline__ int wave_sum_int(int x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ int clamp_len(int len, int cap) { return len < 0 ? 0 : (len > cap ? cap : len); }

__device__ __forceinline__ int pairs_of(int len) { return ((len + kPage - 1) / kPage + 1) >> 1; }

// Window geometry: a window covers at most kPairs pairs (2 kPairs blocks),
// and its buffer in LDS holds the block-table entries, the tags (one dword
// each), the sequence's boundaries, then the G query rows of the KV head.
// The 8-bit two-slot ring uses half-size windows: its workgroup then needs
// 20,272 B of LDS instead of 21,040 B at G = 4, so 8 instead of 7 fit a CU
// (its BASE path is bound by latency, and the eighth wave shortens it).
template <bool SMALL>
struct WinGeo {
  static constexpr int kPairs = SMALL ? 16 : 32;
  static constexpr int kBt = 0, kTags = 8 * kPairs, kBounds = 16 * kPairs, kQ = 16 * kPairs + 16;
};
template <int G, bool SMALL> constexpr int win_bytes() { return WinGeo<SMALL>::kQ + G * 2 * kHeadDim; }

// Position in the flattened (sequence, KV head, pair) space.
struct Walker {
  int s, kvh, j;        // sequence, KV head, pair index of the next window
  int np, nblk, len;    // of sequence s
  int seq_base;         // flattened offset of (s, 0, 0)
  int g;                // flattened offset of (s, kvh, j)
  int lens_base, lens_lane;
};

struct Window {
  int s, kvh, len, b0, b1, j0, j1, np, seq_base;
  bool piece_start, piece_end;
};

template <int G, bool ELASTIC, int NSLOT, bool SMALL>
struct alignas(16) DecodeSmem {
  char ring[NSLOT][kSlotBytes];
  char win[NSLOT + 1][win_bytes<G, SMALL>()];
};

// ---------------------------------------------------------------------------
// Decode kernel: workgroup w streams a range of pairs of the flattened
// (sequence, KV head, pair) space, [w*chunk, (w+1)*chunk) where chunk =
// ceil(T / grid) (at least a.min_chunk) and T counts every pair of every
// (sequence, KV head); with a.heavy > 0 the first a.heavy ranges are
// a.heavy_permille / 1000 times the mean and the others share the rest.
// A (sequence, KV head) that lies wholly inside one range is written out
// directly; one cut by range ends leaves one partial per piece,
// and the last piece to arrive merges them (after its stream has ended).
// ---------------------------------------------------------------------------
template <typename T, int G, bool ELASTIC, int NSLOT, bool F8, bool FUSED>
__global__ __launch_bounds__(64) void decode_kernel(DecodeArgs a) {
  constexpr bool kSmallWin = F8 && NSLOT == 2;
  using Geo = WinGeo<kSmallWin>;
  constexpr int kWinPairs = Geo::kPairs, kWinBt = Geo::kBt, kWinTags = Geo::kTags, kWinBounds = Geo::kBounds,
                kWinQ = Geo::kQ;
  __shared__ DecodeSmem<G, ELASTIC, NSLOT, kSmallWin> sm;
  // query groups of at most 8 heads hold each head in two MFMA columns
  // (n and n + G): P's 16-bit head and remainder accumulate side by side
  constexpr bool kStack = 2 * G <= 16;
  constexpr int kQCols = kStack ? 2 * G : G;
  const int lane = threadIdx.x;
  const int n = lane & 15;
  const int g = lane >> 4;
  const int hkv = a.num_kv_heads;
  const int B = a.batch;
  EKV_TL(const uint64_t tl_start = __builtin_amdgcn_s_memrealtime(); uint64_t tl_first = 0; uint64_t tl_stream = 0;)

  // ---- the range of this workgroup -------------------------------------
  const int len0 = lane < B ? clamp_len(a.seq_lens[lane], a.len_cap) : 0;   // kept: sequences 0..63
  int total_pairs = 0;
  for (int c0 = 0; c0 < B; c0 += 512) {
    int np8[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = c0 + 64 * u + lane;
      np8[u] = pairs_of(idx < 64 ? len0 : (idx < B ? clamp_len(a.seq_lens[idx], a.len_cap) : 0));
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) total_pairs += __builtin_amdgcn_readfirstlane(wave_sum_int(np8[u]));
  }
  const int T_all = hkv * total_pairs;
  if (blockIdx.x == 0) {   // empty sequences: zero output
    for (int c0 = 0; c0 < B; c0 += 64) {
      const int idx = c0 + lane;
      uint64_t empty = __builtin_amdgcn_ballot_w64(idx < B && clamp_len(a.seq_lens[idx], a.len_cap) == 0);
      while (empty) {
        const int s0 = c0 + __builtin_ctzll(empty);
        empty &= empty - 1;
        for (int e = lane; e < a.num_q_heads * kHeadDim / 2; e += 64)
          store_pair<T>(a.out, (size_t)s0 * a.num_q_heads * kHeadDim + 2 * e, 0.f, 0.f, a.out_fp32);
      }
    }
  }
  // Ranges: `heavy` leading workgroups stream r_heavy pairs each, the others r_light
  // (equal ranges when heavy is 0 or the work is at the minimum range).
  const int grid = (int)gridDim.x;
  int r_heavy = max(a.min_chunk, (T_all + grid - 1) / grid), r_light = r_heavy, heavy = 0;
  if (a.heavy > 0 && a.heavy < grid && (T_all + grid - 1) / grid > a.min_chunk) {
    heavy = a.heavy;
    r_heavy = max(1, (int)(((long long)T_all * a.heavy_permille + 1000LL * grid - 1) / (1000LL * grid)));
    const long long rest = (long long)T_all - (long long)heavy * r_heavy;
    r_light = rest > 0 ? (int)((rest + (grid - heavy) - 1) / (grid - heavy)) : 1;
  }
  const long long heavy_end = (long long)heavy * r_heavy;
  auto range_start = [&](int w) -> long long {
    return w < heavy ? (long long)w * r_heavy : heavy_end + (long long)(w - heavy) * r_light;
  };
  auto range_of = [&](int pos) -> int {   // the workgroup whose range holds pair pos
    return pos < heavy_end ? pos / r_heavy : heavy + (int)((pos - heavy_end) / r_light);
  };
  if (range_start((int)blockIdx.x) >= T_all) return;
  const int start = (int)range_start((int)blockIdx.x);
  const int end = (int)min((long long)T_all, range_start((int)blockIdx.x + 1));

  Walker w0;
  {
    int cum = 0;
    for (int c0 = 0;; c0 += 64) {
      const int idx = c0 + lane;
      const int len = c0 == 0 ? len0 : (idx < B ? clamp_len(a.seq_lens[idx], a.len_cap) : 0);
      const int np = pairs_of(len);
      const int incl = wave_incl_scan(np, lane);
      const uint64_t hit = __builtin_amdgcn_ballot_w64(hkv * (cum + incl) > start);
      if (hit) {
        const int l0 = __builtin_ctzll(hit);
        w0.s = c0 + l0;
        w0.len = __builtin_amdgcn_readlane(len, l0);
        w0.np = __builtin_amdgcn_readlane(np, l0);
        w0.seq_base = hkv * (cum + __builtin_amdgcn_readlane(incl, l0) - w0.np);
        w0.lens_base = c0;
        w0.lens_lane = len;
        break;
      }
      cum += __builtin_amdgcn_readlane(incl, 63);
    }
    w0.nblk = (w0.len + kPage - 1) / kPage;
    const int off = start - w0.seq_base;
    w0.kvh = off / w0.np;
    w0.j = off - w0.kvh * w0.np;
    w0.g = start;
  }

  auto next_window = [&](Walker& w) -> Window {
    Window x;
    x.s = w.s;
    x.kvh = w.kvh;
    x.len = w.len;
    x.np = w.np;
    x.seq_base = w.seq_base;
    x.j0 = w.j;
    x.j1 = min(min(w.np, w.j + kWinPairs), w.j + (end - w.g));
    x.b0 = 2 * x.j0;
    x.b1 = min(w.nblk, 2 * x.j1);
    x.piece_start = (x.j0 == 0) || (w.g == start);
    w.g += x.j1 - x.j0;
    w.j = x.j1;
    x.piece_end = (x.j1 == w.np) || (w.g == end);
    if (w.j == w.np && w.g < end) {
      w.j = 0;
      if (++w.kvh == hkv) {
        w.kvh = 0;
        w.seq_base += hkv * w.np;
        do {   // the next sequence that has tokens (one exists: w.g < end)
          ++w.s;
          if (w.s - w.lens_base >= 64) {
            w.lens_base = w.s;
            w.lens_lane = w.s + lane < B ? clamp_len(a.seq_lens[w.s + lane], a.len_cap) : 0;
          }
          w.len = __builtin_amdgcn_readlane(w.lens_lane, w.s - w.lens_base);
        } while (w.len == 0);
        w.np = pairs_of(w.len);
        w.nblk = (w.len + kPage - 1) / kPage;
      }
    }
    return x;
  };

  // ---- per-window metadata by direct-to-LDS loads ------------------------
  const bool have_bounds = ELASTIC && a.bounds != nullptr;
  const bool have_tags = ELASTIC && a.tags != nullptr;
  constexpr int kQInstr = (G * 2 * kHeadDim + 1023) / 1024;
  const int win_ops = 1 + (have_tags ? 1 : 0) + (have_bounds ? 1 : 0) + kQInstr;
  int ops = 0;   // direct-to-LDS load instructions issued so far (stores are not counted)

  auto dma_window = [&](const Window& x, int slot) {
    char* wb = sm.win[slot];
    const int nb = x.b1 - x.b0;
    const size_t row = (size_t)x.s * a.max_blocks + x.b0;
    // (scalar base + 32-bit lane offset: no 64-bit per-lane address stays
    // live across the stream for these once-per-window loads)
    if (lane < nb)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(reinterpret_cast<const char*>(a.bt + row) + lane_offset(4 * lane)),
                                       (lds_ptr)(wb + kWinBt), 4, 0, 0);
    if (have_tags && lane < nb)
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(reinterpret_cast<const char*>(a.tags + row) + lane_offset(lane)),
                                       (lds_ptr)(wb + kWinTags), 1, 0, 0);
    if (have_bounds && lane < 2)
      __builtin_amdgcn_global_load_lds(
          static_cast<const void*>(reinterpret_cast<const char*>(a.bounds + 2 * x.s) + lane_offset(4 * lane)),
          (lds_ptr)(wb + kWinBounds), 4, 0, 0);
    const char* qsrc = reinterpret_cast<const char*>(a.q) + ((size_t)x.s * a.num_q_heads + (size_t)x.kvh * G) * 2 * kHeadDim;
#pragma unroll
    for (int r = 0; r < kQInstr; ++r)
      if (64 * r + lane < G * 16)
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(qsrc + lane_offset(16 * (64 * r + lane))),
                                         (lds_ptr)(wb + kWinQ + 1024 * r), 16, 0, 0);
    ops += win_ops;
  };

  struct ModeInfo {
    int base_lo, base_hi;
    bool use_tags;
  };
  // read a window's block-table entry / tag (per lane) and mode description
  auto window_mode = [&](const char* wb, int& tag_lane) -> ModeInfo {
    ModeInfo m{0, 0, false};
    if constexpr (ELASTIC) {
      int b0 = -1, b1 = -1;
      if (have_bounds) {
        const int2 bb = *reinterpret_cast<const int2*>(wb + kWinBounds);
        b0 = __builtin_amdgcn_readfirstlane(bb.x);
        b1 = __builtin_amdgcn_readfirstlane(bb.y);
      }
      if (b0 >= 0) {
        m.base_lo = 2 * b0;
        m.base_hi = 2 * b1;
      } else if (have_tags) {
        m.use_tags = true;
        tag_lane = *reinterpret_cast<const int*>(wb + kWinTags + 4 * lane);
      }
    }
    return m;
  };
  auto block_is_base = [&](const ModeInfo& m, int tag_lane, int b0, int blk) -> bool {
    if constexpr (!ELASTIC) return false;
    else return m.use_tags ? (__builtin_amdgcn_readlane(tag_lane, blk - b0) != 0)
                           : (blk >= m.base_lo && blk < m.base_hi);
  };

  // ---- fused append ------------------------------------------------------
  // The newest token of a sequence (position len - 1) takes its K / V rows
  // from k_new / v_new.  Its block is TARGET (a caller's invariant; a BASE
  // block is left as it is).  The issue side follows that block's tile loads
  // with two loads of the new rows into the same slot, at the token's row:
  // loads return in order, so they overwrite the pool's old row there.  The
  // consume side, which owns the block's (sequence, KV head) tile in this
  // launch, writes the rows from LDS to the pool.  One row is 2 x 128 words
  // (16 lanes x 16 B) or, for 8-bit pools, 2 x 128 bytes (8 lanes x 16 B).
  constexpr bool fused = FUSED;   // (a separate instance: the plain decode keeps none of this code)
  constexpr int kRowBytes = F8 ? kHeadDim : 2 * kHeadDim;
  constexpr int kRowLanes = kRowBytes / 16;
  auto patched = [&](int len, int blk, bool base) -> bool { return fused && !base && blk == (len - 1) / kPage; };
  // chunk of the row that lane i moves: the one the slot's swizzle puts at i
  auto row_chunk = [&](int t) -> int { return F8 ? (lane ^ tau(t)) : (lane ^ t); };
  auto dma_new_row = [&](int s, int kvh, int t, char* k_row, char* v_row) {
    if (lane < kRowLanes) {
      const size_t off = ((size_t)s * hkv + kvh) * kRowBytes + 16 * row_chunk(t);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(static_cast<const char*>(a.k_new) + off), (lds_ptr)k_row,
                                       16, 0, 0);
      __builtin_amdgcn_global_load_lds(static_cast<const void*>(static_cast<const char*>(a.v_new) + off), (lds_ptr)v_row,
                                       16, 0, 0);
    }
    ops += 2;
  };
  // the rows, from the slot (k_row, v_row: their LDS addresses) to the pool
  auto store_new_row = [&](int phys, int kvh, int t, const char* k_row, const char* v_row) {
    if (lane < kRowLanes) {
      const u32x4 kr = *reinterpret_cast<const u32x4*>(k_row + 16 * lane);
      const u32x4 vr = *reinterpret_cast<const u32x4*>(v_row + 16 * lane);
      constexpr size_t kTileP = F8 ? kTileBytes / 2 : kTileBytes;
      char* dst = static_cast<char*>(a.pool_out) + (size_t)phys * 2 * hkv * kTileP + (size_t)kvh * kTileP +
                  (size_t)t * kRowBytes + 16 * row_chunk(t);
      *reinterpret_cast<u32x4*>(dst) = kr;
      *reinterpret_cast<u32x4*>(dst + (size_t)hkv * kTileP) = vr;
    }
  };

  // per-lane LDS read offsets inside a slot (see the swizzle above)
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
  const DmaOffsets dma = dma_offsets(lane);
  // 8-bit format: nibble-tile load offsets and nibble-operand read offsets
  constexpr int kUnit = kTileBytes;   // 4 KiB
  uint32_t nib[2], rv4[4], rk4 = 0;
  if constexpr (F8) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int p = 64 * r + lane, t = (p >> 2) & 15;
      nib[r] = (p >> 6) * (kTileBytes / 4) + t * (kHeadDim / 2) + 16 * ((p & 3) ^ ((t >> 2) & 3));
    }
    rk4 = n * (kHeadDim / 2) + 16 * (g ^ ((n >> 2) & 3));
#pragma unroll
    for (int i = 0; i < 4; ++i) rv4[i] = (4 * g + i) * (kHeadDim / 2) + 16 * ((n >> 2) ^ g) + 4 * (n & 3);
  }

  // a (plane, head) tile: 4 KiB of 16-bit words, or 2 KiB of bytes (F8)
  constexpr int kTile = F8 ? kTileBytes / 2 : kTileBytes;
  const size_t block_bytes = (size_t)2 * hkv * kTile;
  const size_t v_off = (size_t)hkv * kTile;

  // ---- issue side ------------------------------------------------------
  Walker iwk = w0;
  Window icur = next_window(iwk);
  dma_window(icur, 0);
  const int ops_w0 = ops;
  bool i_has_next = iwk.g < end;
  Window inext = icur;
  int ops_inext = 0;
  if (i_has_next) {
    inext = next_window(iwk);
    dma_window(inext, 1);
    ops_inext = ops;
  }
  const int ops_prologue = ops;
  int iw_idx = 0;
  wait_vm<NSLOT - 1>(ops - ops_w0);
  int bt_lane = *reinterpret_cast<const int*>(sm.win[0] + kWinBt + 4 * lane);
  int itag = 0;
  ModeInfo imode = window_mode(sm.win[0], itag);
  int ib = icur.b0;
  int islot = 0;
  bool issue_done = false;
  int n_issued = 0, n_consumed = 0;   // ring slots

  // enter the next window (its metadata was requested one window ago)
  auto enter_issue_window = [&]() {
    icur = inext;
    ++iw_idx;
    const int ws = iw_idx % (NSLOT + 1);
    wait_vm<NSLOT - 1>(ops - ops_inext);
    bt_lane = *reinterpret_cast<const int*>(sm.win[ws] + kWinBt + 4 * lane);
    imode = window_mode(sm.win[ws], itag);
    i_has_next = iwk.g < end;
    if (i_has_next) {
      inext = next_window(iwk);
      dma_window(inext, (iw_idx + 1) % (NSLOT + 1));
      ops_inext = ops;
    }
    ib = icur.b0;
  };

  auto issue_slot = [&]() {
    if (ib >= icur.b1) enter_issue_window();
    const bool base = block_is_base(imode, itag, icur.b0, ib);
    int phys = __builtin_amdgcn_readlane(bt_lane, ib - icur.b0);
    phys = (unsigned)phys < (unsigned)a.num_blocks ? phys : 0;   // never leave the pool
    const char* src = reinterpret_cast<const char*>(a.pool) + (size_t)phys * block_bytes + (size_t)icur.kvh * kTile;
    char* dst = sm.ring[islot];
    if constexpr (F8) {
      char* ring0 = &sm.ring[0][0];
      char* dk = ring0 + kUnit * islot;
      char* dv = ring0 + kUnit * (islot + 1 == 2 * NSLOT ? 0 : islot + 1);
      int units = 2;
      if (base) {
        dma_nibbles(src, nib, dk);
        dma_nibbles(src + v_off, nib, dk + kTileBytes / 2);
        ops += 4;
        ib += 2;
        units = 1;
      } else {
        const bool pair = ib + 1 < icur.b1;
        if (pair) {
          // a whole TARGET pair: member m's rows from its own block, in the
          // layout of a 16-bit packed BASE pair (bytes, member-major)
          int phys1 = __builtin_amdgcn_readlane(bt_lane, ib + 1 - icur.b0);
          phys1 = (unsigned)phys1 < (unsigned)a.num_blocks ? phys1 : 0;
          const char* src1 = reinterpret_cast<const char*>(a.pool) + (size_t)phys1 * block_bytes +
                             (size_t)icur.kvh * kTile;
          dma_pair_bytes(src, src1, dma.base, dk);
          dma_pair_bytes(src + v_off, src1 + v_off, dma.base, dv);
          ops += 8;
        } else {
          // the sequence's last block, alone: member 0 only
          dma_member0_bytes(src, dma.base, dk);
          dma_member0_bytes(src + v_off, dma.base, dv);
          ops += 4;
        }
        for (int m = 0; m < (pair ? 2 : 1); ++m)
          if (patched(icur.len, ib + m, false)) {
            const int t = (icur.len - 1) % kPage;
            dma_new_row(icur.s, icur.kvh, t, dk + m * (kTileBytes / 2) + t * kRowBytes,
                        dv + m * (kTileBytes / 2) + t * kRowBytes);
          }
        ib += pair ? 2 : 1;
      }
      islot += units;
      if (islot >= 2 * NSLOT) islot -= 2 * NSLOT;
      n_issued += units;
    } else {
      if (base) {
        dma_tile(src, dma.base, dst);
        dma_tile(src + v_off, dma.base, dst + kTileBytes);
      } else {
        dma_tile(src, dma.tgt, dst);
        dma_tile(src + v_off, dma.tgt, dst + kTileBytes);
      }
      ops += 8;
      if (patched(icur.len, ib, base)) {
        const int t = (icur.len - 1) % kPage;
        dma_new_row(icur.s, icur.kvh, t, dst + t * kRowBytes, dst + kTileBytes + t * kRowBytes);
      }
      ib += base ? 2 : 1;
      islot = islot + 1 == NSLOT ? 0 : islot + 1;
      ++n_issued;
    }
    issue_done = ib >= icur.b1 && !i_has_next;
  };

  // ---- consume side ----------------------------------------------------
  Walker cwk = w0;
  Window ccur = next_window(cwk);
  int cw_idx = 0;
  int c_ops = ops_prologue;     // instructions issued up to and including the slot being consumed
  int ctag = 0;
  ModeInfo cmode = window_mode(sm.win[0], ctag);
  // The softmax takes c = |scale| log2(e); a negative scale negates the
  // query instead (a sign flip of each 16-bit word, exact).
  const float c_scale = fabsf(a.scale_log2);
  const uint32_t q_sign = a.scale_log2 < 0.f ? 0x80008000u : 0u;
  u32x4 qop[4];
  auto load_q = [&](const char* wb) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      qop[k] = (n < kQCols)
                   ? (*reinterpret_cast<const u32x4*>(wb + kWinQ + (n % G) * 2 * kHeadDim + 16 * (4 * g + k)) ^ q_sign)
                   : u32x4{0u, 0u, 0u, 0u};
      if constexpr (F8) qop[k] = q_words_x4(qop[k]);
    }
  };
  load_q(sm.win[0]);
  // Fused append: the physical block of the newest token's block when it
  // lies in the consume side's window, read when the side enters the window
  // (like its tags and queries).  A window's buffer can be refilled for a
  // later window while the consume side still works in it (the 8-bit ring
  // holds units of three windows, one per buffer, when windows are one unit
  // long), so nothing is read from it after entry.
  auto newest_block = [&](const char* wb) -> int {
    if constexpr (!fused) return 0;
    const int nb = (ccur.len - 1) / kPage;
    if (nb < ccur.b0 || nb >= ccur.b1) return 0;
    const int phys = __builtin_amdgcn_readfirstlane(*reinterpret_cast<const int*>(wb + kWinBt + 4 * (nb - ccur.b0)));
    return (unsigned)phys < (unsigned)a.num_blocks ? phys : 0;
  };
  int c_new_phys = newest_block(sm.win[0]);
  int cb = ccur.b0;
  int cslot = 0;
  int piece_j0 = ccur.j0;

  SplitState st;
  auto reset = [&]() {
#pragma unroll
    for (int j = 0; j < 8; ++j) st.o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    st.m = -__builtin_inff();
    st.l = 0.f;
  };
  reset();

  // partial pieces whose merge counter is bumped after the stream (at most 2)
  int pend_n = 0;
  size_t pend_head0[2] = {0, 0};
  int pend_wfirst[2] = {0, 0}, pend_odd[2] = {0, 0}, pend_pieces[2] = {0, 0};

  auto finalize_piece = [&]() {
    if constexpr (kStack) stacked_sum<G>(st);
    const float l = head_sum(st.l);
    const size_t head0 = (size_t)ccur.s * a.num_q_heads + (size_t)ccur.kvh * G;
    const int first = ccur.seq_base + ccur.kvh * ccur.np;
    const int w_first = range_of(first), w_last = range_of(first + ccur.np - 1);
    const int pieces = w_last - w_first + 1;
    if (pieces == 1) {
      if (n < G) {
        const float inv = 1.0f / l;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          store_row8<T>(a.out, (head0 + n) * kHeadDim + 32 * g + 8 * r,
                        f32x4{st.o[0][r], st.o[1][r], st.o[2][r], st.o[3][r]} * inv,
                        f32x4{st.o[4][r], st.o[5][r], st.o[6][r], st.o[7][r]} * inv, a.out_fp32);
      }
    } else {
      // this workgroup's slot for the piece: 2w if the (sequence, KV head)
      // contains its first pair, else 2w + 1
      const size_t slot = (size_t)(2 * (int)blockIdx.x + (first > start ? 1 : 0));
      const size_t row = slot * G + n;
      if (n < G) {
        // chunk ci = 2 r + half of this lane at chunk ci * 4G + n + G g of the slot
        float* dst = a.ws_o + slot * G * kHeadDim + 4 * (n + G * g);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          store_agent_f4(dst + (2 * r) * 16 * G, f32x4{st.o[0][r], st.o[1][r], st.o[2][r], st.o[3][r]});
          store_agent_f4(dst + (2 * r + 1) * 16 * G, f32x4{st.o[4][r], st.o[5][r], st.o[6][r], st.o[7][r]});
        }
        if (g == 0) store_agent_f2(a.ws_ml + 2 * row, st.m, l);
      }
      pend_head0[pend_n] = head0;
      pend_wfirst[pend_n] = w_first;
      pend_odd[pend_n] = first > range_start(w_first) ? 1 : 0;
      pend_pieces[pend_n] = pieces;
      ++pend_n;
    }
  };

  // ring capacity: NSLOT slots, or (8-bit) 2 NSLOT units of which a slot takes up to two
  auto ring_has_room = [&]() {
    return F8 ? n_issued - n_consumed + 2 <= 2 * NSLOT : n_issued - n_consumed < NSLOT;
  };
#pragma unroll
  for (int k = 0; k < (F8 ? 2 * NSLOT - 2 : NSLOT - 1); ++k)
    if (!issue_done && ring_has_room()) issue_slot();

  while (true) {
    // keep the ring full
#pragma unroll
    for (int u = 0; u < 2; ++u)
      if (!issue_done && ring_has_room()) issue_slot();
    if constexpr (F8) {
      // one slot: a BASE pair (nibbles), a TARGET pair, or the lone last block
      const bool base = block_is_base(cmode, ctag, ccur.b0, cb);
      const bool lone = !base && cb + 1 >= ccur.b1;
      c_ops += (base || lone) ? 4 : 8;
      int new_member = -1;   // fused append: the member holding the newest token
      if (!base)
        for (int m = 0; m < (lone ? 1 : 2); ++m)
          if (patched(ccur.len, cb + m, false)) new_member = m;
      if (new_member >= 0) c_ops += 2;
      wait_vm4(ops - c_ops);
      EKV_TL(if (!tl_first) tl_first = __builtin_amdgcn_s_memrealtime();)
      const char* ring0 = &sm.ring[0][0];
      const char* kb = ring0 + kUnit * cslot;
      const char* vb = ring0 + kUnit * (cslot + 1 == 2 * NSLOT ? 0 : cslot + 1);
      if (new_member >= 0) {
        const int t = (ccur.len - 1) % kPage;
        const int mo = new_member * (kTileBytes / 2) + t * kRowBytes;
        store_new_row(c_new_phys, ccur.kvh, t, kb + mo, vb + mo);
      }
      f32x4 sc[2];
      PvOps<kStack> pvo;
      if (base) {
        // nibbles straight to 16-bit operand words (a BASE pair is two full
        // blocks: no tail to clear)
        NibPlanes pv[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const char* mb = kb + m * (kTileBytes / 4);
          const u32x4 kn = *reinterpret_cast<const u32x4*>(mb + rk4);
          u32x4 kw[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) kw[q] = nib_words_x4(kn[q]);
          sc[m] = qk_scores<T, false>(kw, qop);
#pragma unroll
          for (int i = 0; i < 4; ++i)
            pv[m][i] = nib_planes(*reinterpret_cast<const uint32_t*>(mb + kTileBytes / 2 + rv4[i]));
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const u32x2 a0 = nib_v_operand(pv[0], j), a1 = nib_v_operand(pv[1], j);
          if constexpr (kStack) pvo.v[j] = u32x4{a0.x, a0.y, a1.x, a1.y};
          else {
            pvo.v[0][j] = a0;
            pvo.v[1][j] = a1;
          }
        }
      } else {
        // (only .xy of each V operand is loaded: the byte path reads no
        // more, and zero .zw lets the tail clearing below fold to nothing there)
        u32x4 k[2][4], v[2][4] = {};
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const char* mb = kb + m * (kTileBytes / 2);
          const u32x4 k0 = *reinterpret_cast<const u32x4*>(mb + rk_b[0]);
          const u32x4 k1 = *reinterpret_cast<const u32x4*>(mb + rk_b[1]);
          k[m][0].xy = k0.xy;
          k[m][1].xy = k0.zw;
          k[m][2].xy = k1.xy;
          k[m][3].xy = k1.zw;
          const char* mv = vb + m * (kTileBytes / 2) - kTileBytes;   // rv_b counts from the K tile
#pragma unroll
          for (int i = 0; i < 4; ++i) v[m][i].xy = *reinterpret_cast<const u32x2*>(mv + rv_b[i]);
          f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int st = 0; st < 4; ++st) s = Mma<T>::qk(byte_words_x4(k[m][st].xy), qop[st], s);
          sc[m] = s;
        }
        zero_tail_v<2>(v, cb * kPage, ccur.len, g);
        pv_operands<true, 2>(v, pvo);
      }
      const bool tail = cb * kPage + 2 * kPage > ccur.len;
      pv_step<T, G>(st, sc, pvo, cb * kPage, ccur.len, tail, c_scale, g, n);
      cb += lone ? 1 : 2;
      const int units = base ? 1 : 2;
      n_consumed += units;
      cslot += units;
      if (cslot >= 2 * NSLOT) cslot -= 2 * NSLOT;
    } else {
    c_ops += 8;
    const bool base0 = block_is_base(cmode, ctag, ccur.b0, cb);
    const bool new0 = patched(ccur.len, cb, base0);   // fused append: the newest token is in block cb
    if (new0) c_ops += 2;
    wait_vm<NSLOT - 1>(ops - c_ops);
    EKV_TL(if (!tl_first) tl_first = __builtin_amdgcn_s_memrealtime();)
    const char* sb = sm.ring[cslot];
    const int t_new = (ccur.len - 1) % kPage;
    if (new0) store_new_row(c_new_phys, ccur.kvh, t_new, sb + t_new * kRowBytes, sb + kTileBytes + t_new * kRowBytes);
    // Each kind of step leaves its scores and PV operands here; one softmax
    // and PV call follows for all of them.  A step of one TARGET block (the
    // lone last block, or any block with a ring of fewer than 4 slots) masks
    // the empty second group through lim.
    f32x4 sc[2];
    PvOps<kStack> pvo;
    int step_blocks = 2, step_slots = 1;
    if (base0) {
      // one packed pair: member 0 = logical block cb, member 1 = cb + 1
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
        sc[m] = qk_scores<T, true>(k[m], qop);
      }
      pv_operands<true, 2>(v, pvo);
    } else if (NSLOT >= 4 && cb + 1 < ccur.b1) {
      // two TARGET blocks (the two members of a pair, in consecutive slots):
      // one softmax step over 32 tokens, two independent QK chains
      const int cslot2 = cslot + 1 == NSLOT ? 0 : cslot + 1;
      c_ops += 8;
      const bool new1 = patched(ccur.len, cb + 1, false);
      if (new1) c_ops += 2;
      wait_vm<NSLOT - 2>(ops - c_ops);
      const char* sb2 = sm.ring[cslot2];
      if (new1)
        store_new_row(c_new_phys, ccur.kvh, t_new, sb2 + t_new * kRowBytes,
                      sb2 + kTileBytes + t_new * kRowBytes);
      u32x4 k[2][4], v[2][4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        k[0][q] = *reinterpret_cast<const u32x4*>(sb + rk_t[q]);
        k[1][q] = *reinterpret_cast<const u32x4*>(sb2 + rk_t[q]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[0][i] = *reinterpret_cast<const u32x4*>(sb + rv_t[i]);
        v[1][i] = *reinterpret_cast<const u32x4*>(sb2 + rv_t[i]);
      }
      sc[0] = qk_scores<T, false>(k[0], qop);
      sc[1] = qk_scores<T, false>(k[1], qop);
      zero_tail_v<2>(v, cb * kPage, ccur.len, g);
      pv_operands<false, 2>(v, pvo);
      step_slots = 2;
    } else {
      u32x4 k[4], v[1][4];
#pragma unroll
      for (int q = 0; q < 4; ++q) k[q] = *reinterpret_cast<const u32x4*>(sb + rk_t[q]);
#pragma unroll
      for (int i = 0; i < 4; ++i) v[0][i] = *reinterpret_cast<const u32x4*>(sb + rv_t[i]);
      sc[0] = qk_scores<T, false>(k, qop);
      sc[1] = f32x4{0.f, 0.f, 0.f, 0.f};
      zero_tail_v<1>(v, cb * kPage, ccur.len, g);
      pv_operands<false, 1>(v, pvo);
      step_blocks = 1;
    }
    const int lim = step_blocks == 1 ? min(ccur.len, cb * kPage + kPage) : ccur.len;
    const bool mask = step_blocks == 1 || cb * kPage + 2 * kPage > ccur.len;
    pv_step<T, G>(st, sc, pvo, cb * kPage, lim, mask, c_scale, g, n);
    cb += step_blocks;
    n_consumed += step_slots;
    cslot += step_slots;
    if (cslot >= NSLOT) cslot -= NSLOT;
    }   // 16-bit TARGET
    if (cb < ccur.b1) continue;
    // window finished
    if (ccur.piece_end) finalize_piece();
    if (cwk.g >= end) break;
    ccur = next_window(cwk);
    ++cw_idx;
    if (cwk.g < end) c_ops += win_ops;   // the issue side requested the window after this one
    const char* wb = sm.win[cw_idx % (NSLOT + 1)];
    cmode = window_mode(wb, ctag);
    load_q(wb);
    c_new_phys = newest_block(wb);
    if (ccur.piece_start) {
      reset();
      piece_j0 = ccur.j0;
    }
    cb = ccur.b0;
  }
  (void)piece_j0;
  EKV_TL(tl_stream = __builtin_amdgcn_s_memrealtime();
         auto tl_write = [&]() {
           if (lane == 0 && blockIdx.x < 8192) {
             uint64_t* r = g_timeline + 8 * blockIdx.x;
             r[0] = tl_start; r[1] = tl_first; r[2] = tl_stream; r[3] = __builtin_amdgcn_s_memrealtime();
             r[4] = (uint64_t)(end - start); r[5] = (uint64_t)pend_n;
             // XCC_ID (hwreg 20, bits 0..15); HW_ID (hwreg 4: wave slot, SIMD, CU, SH, SE) in bits 32..63
             r[6] = (uint64_t)__builtin_amdgcn_s_getreg(30740) | ((uint64_t)__builtin_amdgcn_s_getreg(63492) << 32);
             r[7] = 1;
           }
         };)

  // ---- merges ----------------------------------------------------------
  if (pend_n == 0) {
    EKV_TL(tl_write();)
    return;
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // partials have landed before they are counted
  // both counters are bumped before either result is awaited
  uint32_t prev0 = 0u, prev1 = 0u;
  if (lane == 0) {
    prev0 = __hip_atomic_fetch_add(a.counters + piece_slot(pend_wfirst[0], pend_odd[0], 0), 1u, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    if (pend_n > 1)
      prev1 = __hip_atomic_fetch_add(a.counters + piece_slot(pend_wfirst[1], pend_odd[1], 0), 1u, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
  }
  for (int k = 0; k < pend_n; ++k) {
    uint32_t* counter = a.counters + piece_slot(pend_wfirst[k], pend_odd[k], 0);
    if (__builtin_amdgcn_readfirstlane(k == 0 ? prev0 : prev1) != (uint32_t)(pend_pieces[k] - 1)) continue;
    asm volatile("" ::: "memory");
    if (lane == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (pend_pieces[k] <= 64) merge_splits<T, G>(a, pend_head0[k], pend_pieces[k], pend_wfirst[k], pend_odd[k], lane);
    else
      for (int h = 0; h < G; ++h)
        merge_head_serial<T, G>(a, pend_head0[k] + h, h, pend_pieces[k], pend_wfirst[k], pend_odd[k], lane);
  }
  EKV_TL(tl_write();)
}

// Workgroups that fit on the device at once for a kernel (one wave each):
// compute units and workgroups per compute unit, cached per device and
// kernel instance (occupancy does not change).
struct Residency {
  int cus = 0, per_cu = 0;
  int total() const { return cus * per_cu; }
};
template <typename K>
Residency residency(K kernel, std::atomic<int>* cache) {
  Residency r;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return r;
  const int packed = cache[dev].load(std::memory_order_relaxed);
  if (packed > 0) {
    r.cus = packed >> 8;
    r.per_cu = packed & 255;
    return r;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return r;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 64, 0) != hipSuccess) return r;
  if (cus <= 0 || per_cu <= 0 || per_cu > 255) return r;
  r.cus = cus;
  r.per_cu = per_cu;
  cache[dev].store((cus << 8) | per_cu, std::memory_order_relaxed);
  return r;
}

// Range weighting for instances that hold two waves on every SIMD: the
// first 4 x CUs workgroups of a full grid each take a SIMD's first slot and
// are issued ahead of the second-slot waves, which then stream more slowly;
// with equal ranges the second-slot waves finished ~25 % later (8-bit pool,
// BASE fraction 1).  So the first-slot workgroups take ranges of
// kHeavyPermille / 1000 times the mean and the others share the rest
// (EKV_HEAVY_PERMILLE overrides; 1000 gives equal ranges).
constexpr int kHeavyPermille = 1150;
int heavy_permille() {
  if (const char* env = getenv("EKV_HEAVY_PERMILLE")) return std::max(1000, std::min(1900, atoi(env)));
  return kHeavyPermille;
}

// Launches the instance, or (grid_out != null) only reports the grid it
// would use: the resident workgroups, or fewer when the work is small.
template <typename T, int G, int NSLOT, bool F8>
hipError_t run_slots(const DecodeArgs& a, bool elastic, hipStream_t st, int* grid_out) {
  static std::atomic<int> cache[2][kMaxDevices];
  auto kernel = elastic ? decode_kernel<T, G, true, NSLOT, F8, false> : decode_kernel<T, G, false, NSLOT, F8, false>;
  const Residency res = residency(kernel, cache[elastic ? 1 : 0]);
  if (res.total() <= 0) return hipErrorInvalidDeviceFunction;
  if (grid_out) {   // (the grid of the plain decode; the fused instance has the same registers and LDS)
    const int resident = res.total();
    const long long wanted = (a.pairs_max + a.min_chunk - 1) / a.min_chunk;
    *grid_out = (int)std::max<long long>(1, std::min<long long>(std::min(resident, kMaxDecodeGrid), wanted));
    return hipSuccess;
  }
  if (a.grid <= 0) return hipErrorInvalidValue;
  if (a.k_new)
    kernel = elastic ? decode_kernel<T, G, true, NSLOT, F8, true> : decode_kernel<T, G, false, NSLOT, F8, true>;
  DecodeArgs b = a;
  b.heavy = 0;
  b.heavy_permille = 1000;
  if (res.per_cu == 8 && a.grid == res.total()) {
    b.heavy = 4 * res.cus;
    b.heavy_permille = heavy_permille();
  }
  hipLaunchKernelGGL(kernel, dim3(b.grid), dim3(64), 0, st, b);
  return hipGetLastError();
}

template <typename T, int G, bool F8>
hipError_t run_typed(const DecodeArgs& a, bool elastic, hipStream_t st, int* grid_out) {
  switch (a.slots) {
    case 2: return run_slots<T, G, 2, F8>(a, elastic, st, grid_out);
    case 4: return run_slots<T, G, 4, F8>(a, elastic, st, grid_out);
    default: return run_slots<T, G, 3, F8>(a, elastic, st, grid_out);
  }
}

template <typename T, bool F8>
hipError_t run_group(const DecodeArgs& a, int group, bool elastic, hipStream_t st, int* grid_out) {
  switch (group) {
    case 1: return run_typed<T, 1, F8>(a, elastic, st, grid_out);
    case 2: return run_typed<T, 2, F8>(a, elastic, st, grid_out);
    case 4: return run_typed<T, 4, F8>(a, elastic, st, grid_out);
    case 8: return run_typed<T, 8, F8>(a, elastic, st, grid_out);
    case 16: return run_typed<T, 16, F8>(a, elastic, st, grid_out);
    default: return hipErrorInvalidValue;
  }
}

hipError_t run_dtype(const DecodeArgs& a, int dtype, int group, bool elastic, hipStream_t st, int* grid_out) {
  switch (dtype) {
    case 0: return run_group<Bf16, false>(a, group, elastic, st, grid_out);
    case 1: return run_group<Fp16, false>(a, group, elastic, st, grid_out);
    case 3: return run_group<Fp16, true>(a, group, elastic, st, grid_out);   // E5M2 bytes, FP16 queries
    default: return hipErrorInvalidValue;
  }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int dtype, int group, bool elastic, hipStream_t st) {
  if (a.batch == 0) return hipSuccess;
  return run_dtype(a, dtype, group, elastic, st, nullptr);
}

hipError_t decode_grid(const DecodeArgs& a, int dtype, int group, bool elastic, int* grid) {
  return run_dtype(a, dtype, group, elastic, nullptr, grid);
}

hipError_t launch_zero_u32(uint32_t* p, size_t n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 1024);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace ekv
