// Chunked-prefill attention over a mixed-fidelity paged prefix for gfx950
// (paper §3.2: BASE blocks are read as their high bytes with a zero low
// byte; App. A: a prefill chunk attends its cached prefix and, causally,
// itself).
//
// A workgroup of 4 waves serves one (sequence, KV head, tile of query
// tokens).  Each wave owns 32 query "columns" -- (token, head-in-group)
// pairs -- and the waves share the K/V blocks, which stream through an LDS
// ring by direct-to-LDS loads (each wave loads a quarter of every K and V
// tile; the waves meet at a barrier before a tile is read).
//
// Work unit: 32 keys (two TARGET blocks, or one packed BASE pair, or the
// lone last block).  On 32x32x16 matrix cores:
//   S^T (32 keys x 32 columns) = K (32 x 128) . Q^T, 8 products;
//     lane l holds column l % 32 and keys 8(r/4) + 4(l/32) + r%4, r < 16.
//   online softmax over those 16 scores (+ the partner lane l ^ 32);
//   O^T (128 dims x 32 columns) += V^T . P^T, for P's 16-bit head and its
//     16-bit remainder (P keeps ~16 significant bits), 4 dim tiles x 2
//     key steps x 2.  The P operand of key step k is the lane's own scores
//     r = 8k .. 8k+7, so key index 8(l/32) + i of step k stands for key
//     16k + 8(i/4) + 4(l/32) + i%4; the V^T operand follows the same order.
// V^T operands come straight from LDS with transposing reads: 16-bit
// elements (TARGET) by two ds_read_b64_tr_b16, bytes (BASE) by one
// ds_read_b64_tr_b8 followed by the byte -> high-byte expansion.  Within
// each 16-lane group such a read hands lane j element j of the rows the
// group's lanes point at (row 4a + j/4, element j%4 for 16-bit; row
// 2a + j/8, byte j%8 for 8-bit), so pointing lane 4a + b at key a, dims
// d + 4b .. (resp. lane 2a + b at key a, dims d + 8b ..) gives lane j
// keys a = 0..3 (0..7) of dim d + j.
//
// Column c sees keys p < lim(c) = prefix + (its chunk index) + 1.
// Block-table entries and tags are held in registers per window of 64 blocks.
#include <type_traits>

#include "attn_device.h"

namespace ekv {
namespace {

constexpr int kPfWaves = 4;
constexpr int kPfRing = 4;        // 8 KiB slots
constexpr int kPfCols = 32;       // query columns per wave
constexpr int kPfWindow = 64;     // blocks per metadata window: one per lane

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4v __attribute__((ext_vector_type(4)));
typedef int i32x2v __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4v* lds_i16x4;
typedef __attribute__((address_space(3))) i32x2v* lds_i32x2;

template <typename T> struct Mma32;
template <> struct Mma32<Bf16> {
  static __device__ __forceinline__ f32x16 mma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
  }
};
template <> struct Mma32<Fp16> {
  static __device__ __forceinline__ f32x16 mma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b),
                                                  c, 0, 0, 0);
  }
};

// Two probabilities -> packed 16-bit heads and packed 16-bit remainders
// (head + remainder = p to ~16 significant bits).  bf16: the head is the
// upper half of the fp32 word (truncation), one byte permute for the pair.
template <typename T>
__device__ __forceinline__ void split_p(float p0, float p1, uint32_t& hi, uint32_t& lo);

template <>
__device__ __forceinline__ void split_p<Bf16>(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  const uint32_t x0 = __float_as_uint(p0), x1 = __float_as_uint(p1);
  hi = perm(x1, x0, 0x07060302u);   // upper halves: x0 -> low word, x1 -> high word
  // both remainders rounded to nearest-even in one packed conversion
  const f32x2v rem = {p0 - __uint_as_float(x0 & 0xffff0000u), p1 - __uint_as_float(x1 & 0xffff0000u)};
  lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(rem, bf16x2v));
}
template <>
__device__ __forceinline__ void split_p<Fp16>(float p0, float p1, uint32_t& hi, uint32_t& lo) {
  float b0, b1, dummy;
  const uint16_t h0 = Mma<Fp16>::round(p0, &b0), h1 = Mma<Fp16>::round(p1, &b1);
  const uint16_t e0 = Mma<Fp16>::round(p0 - b0, &dummy), e1 = Mma<Fp16>::round(p1 - b1, &dummy);
  hi = (uint32_t)h0 | ((uint32_t)h1 << 16);
  lo = (uint32_t)e0 | ((uint32_t)e1 << 16);
}

// Prefill's TARGET tile layout: chunk c of token t at position c ^ sw(t),
// sw(t) = 4 (t & 3) + (t >> 2).  The K reads (16 rows at one chunk per
// 16 lanes) and the transposing V reads (4 rows x 4 consecutive chunks per
// 32 lanes) then each touch 16 distinct 16-byte positions of a 256-byte
// bank cycle, with no bank conflict; the decode layout (c ^ t) puts the
// V reads' 4 x 2 chunks of a 16-lane group on only 4 positions.
__device__ __forceinline__ int pf_swizzle(int t) { return 4 * (t & 3) + (t >> 2); }

// Offset in a 4 KiB TARGET tile in HBM of the 16 B that land at LDS chunk p.
__device__ __forceinline__ uint32_t pf_target_offset(int p) {
  const int t = p >> 4, pos = p & 15;
  return t * (2 * kHeadDim) + 16 * (pos ^ pf_swizzle(t));
}

// 8 nibbles (element e in byte e/2, low nibble for even e) -> 8 bytes,
// each nibble in the high half of its byte (an executed 4-bit BASE value).
__device__ __forceinline__ u32x2 widen_nibbles(uint32_t w) {
  const uint32_t even = (w << 4) & 0xF0F0F0F0u, odd = w & 0xF0F0F0F0u;
  return u32x2{perm(odd, even, 0x05010400u), perm(odd, even, 0x07030602u)};
}

// max of three floats.  Written for the compiler, not as inline assembly:
// its operands come straight from the matrix cores, and only the compiler
// inserts the wait states a vector instruction needs before it may read an
// MFMA result (inline assembly would read the registers while the products
// are still being written).
__device__ __forceinline__ float max3(float a, float b, float c) { return __builtin_fmaxf(__builtin_fmaxf(a, b), c); }

// v *= f, written for the compiler: the accumulators come straight from the
// matrix cores, and only the compiler inserts the wait states a vector
// instruction needs before it reads an MFMA result.  (On gfx950 the
// multiplies stay in the accumulators' own registers: no copies on the
// common path that skips the rescale.)
__device__ __forceinline__ void scale_in_place(f32x16& v, float f) {
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] *= f;
}

// Workgroup barrier that also orders this wave's LDS accesses.  On gfx950
// s_barrier does not wait for the wave's outstanding LDS operations, and
// the compiler adds no wait before a bare s_barrier: an LDS write issued
// before it (the widened 8-bit tiles) could land after another wave has
// passed the barrier and read the old bytes, and an LDS read still in
// flight could see a slot that the ring's next load has begun to refill.
// s_waitcnt lgkmcnt(0) completes every LDS access of the wave first.  The
// ring's direct-to-LDS loads are vector memory operations, waited for with
// explicit counts before the barrier that publishes a slot.
__device__ __forceinline__ void barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait until at most 2n of this wave's vector memory instructions are in
// flight (each ring slot costs a wave two loads); 0 <= n < kPfRing, and a
// larger n waits as for kPfRing - 1.
static_assert(kPfRing == 4, "one wait per number of slots that may stay in flight");
__device__ __forceinline__ void wait_slots(int n) {
  n = __builtin_amdgcn_readfirstlane(n);
  if (n >= 3) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
  else if (n == 2) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else if (n == 1) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// At least two waves per SIMD (at most 256 registers): with one, the matrix
// cores idle through every softmax.
// F8: an 8-bit pool (FP8 E5M2 TARGET, 4-bit BASE).  A TARGET pair is
// loaded into a slot in the byte layout of a packed 16-bit BASE pair (member
// m from its own block) and a BASE pair's nibbles are staged and widened
// into that layout, so every unit runs on the byte path with FP16 products.
template <typename T, int G, bool ELASTIC, bool F8>
__global__ __launch_bounds__(64 * kPfWaves) __attribute__((amdgpu_waves_per_eu(2))) void prefill_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) char ring[kPfRing][kSlotBytes];
  __shared__ __attribute__((aligned(16))) char nib[F8 ? kPfRing : 1][F8 ? kTileBytes : 16];
  constexpr int kTileTok = kPfWaves * kPfCols / G;
  const int s = blockIdx.z;
  const int kvh = blockIdx.y;
  const int tile = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int n = lane & 31;     // MFMA column
  const int h = lane >> 5;     // half of the key / head-dim index space
  // query rows of this sequence, clamped into q and out (never leave them)
  const int q0 = min(max(a.cu_q[s], 0), a.total_q);
  const int nq = min(max(a.cu_q[s + 1], q0), a.total_q) - q0;
  const int t_begin = tile * kTileTok;
  if (t_begin >= nq) return;   // uniform over the workgroup
  const int len = max(0, min(a.seq_lens[s], a.max_blocks * kPage));
  const int prefix = len - nq;

  // this lane's query column and its Q^T operands (dims 16k + 8h .. + 7)
  const int col = wave * kPfCols + n;
  const int tq = t_begin + col / G;
  const int head = col % G;
  const bool col_ok = tq < nq;
  const int lim = col_ok ? min(len, prefix + tq + 1) : len;
  // The softmax uses exp2(s * c - m) with c = |scale| log2(e) >= 0; a
  // negative scale is applied by negating Q (exact) instead.
  const float c_scale = fabsf(a.scale_log2);
  const uint32_t q_sign = a.scale_log2 < 0.f ? 0x80008000u : 0u;
  u32x4 qop[8];
  {
    const uint16_t* qrow =
        a.q + ((size_t)(q0 + (col_ok ? tq : 0)) * a.num_q_heads + (size_t)kvh * G + head) * kHeadDim;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      qop[k] = col_ok ? (*reinterpret_cast<const u32x4*>(qrow + 16 * k + 8 * h) ^ q_sign) : u32x4{0u, 0u, 0u, 0u};
  }
  // keys every column of this wave sees (below that no mask is needed)
  const int lim_wave = min(len, prefix + t_begin + wave * kPfCols / G + 1);
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

  // each wave loads quarter `wave` of every K and V tile of a slot, at this
  // LDS address (plus the slot's offset); TARGET tiles in prefill's own
  // swizzle, BASE tiles as in decode
  const DmaOffsets dma = dma_offsets(lane + 64 * wave);
  const uint32_t dma_tgt = pf_target_offset(lane + 64 * wave);
  const uint32_t lds_wave = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_ptr)&ring[0][0] + 1024 * wave);
  // a (plane, head) tile in HBM: 4 KiB of 16-bit words, or 2 KiB of bytes
  constexpr int kTileP = F8 ? kTileBytes / 2 : kTileBytes;
  const size_t block_bytes = (size_t)2 * a.num_kv_heads * kTileP;
  const char* pool = reinterpret_cast<const char*>(a.pool) + (size_t)kvh * kTileP;
  const size_t v_off = (size_t)a.num_kv_heads * kTileP;
  // F8: offset of this lane's 16 B inside its member's tile (waves 0, 1 load
  // member 0, waves 2, 3 member 1), and this wave's share of the staging area
  const uint32_t dma_member = dma.base[0] - (uint32_t)(wave >> 1) * (kTileBytes / 2);
  const uint32_t nib_wave = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_ptr)&nib[0][0] + 512 * wave);
  const int32_t* btrow = a.bt + (size_t)s * a.max_blocks;
  const uint8_t* tagrow = a.tags ? a.tags + (size_t)s * a.max_blocks : nullptr;

  // LDS reads.  K (A operand of S^T): key row m = lane % 32.  V^T: the
  // 16-lane group g16 covers dims 16 (g16 & 1) .. + 15 of each 32-dim tile;
  // within it, position i16 supplies the row address of the transposing read.
  const int t_row = n & 15;
  const int g16 = lane >> 4;
  const int i16 = lane & 15;
  const int tr_a = i16 >> 2, tr_b = i16 & 3;   // 16-bit: key a, dims + 4b
  const int b8_a = i16 >> 1, b8_b = i16 & 1;   // 8-bit: key a, dims + 8b
  // byte offsets inside a slot.  The swizzles only flip the address bits
  // that select the step, so each per-step offset is a per-lane base XOR a
  // constant: K rows kt ^ 32k (16-bit) and kb ^ 16k (bytes) for the 16-dim
  // step k; V^T rows vt[half] ^ 64t (16-bit, per half of the key step) and
  // vb ^ 32t (bytes) for the 32-dim tile t.
  const int f_row = pf_swizzle(t_row);
  const uint32_t off_kt = t_row * (2 * kHeadDim) + 16 * (h ^ (f_row & 1)) + 32 * (f_row >> 1);
  const uint32_t off_kb = (n >> 4) * (kTileBytes / 2) + t_row * kHeadDim + 16 * tau(t_row) + 8 * h;
  uint32_t off_vt[2];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int key = 8 * half + 4 * h + tr_a;
    const int x = 2 * (g16 & 1) + (tr_b >> 1);
    const int f = pf_swizzle(key);
    off_vt[half] = kTileBytes + key * (2 * kHeadDim) + 16 * (x ^ (f & 3)) + 64 * (f >> 2) + 8 * (tr_b & 1);
  }
  const int keyb = 8 * (b8_a >> 2) + 4 * h + (b8_a & 3);
  const uint32_t off_vb =
      kTileBytes + keyb * kHeadDim + 16 * ((g16 & 1) ^ (tau(keyb) & 1)) + 32 * (tau(keyb) >> 1) + 8 * b8_b;

  f32x16 o[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) o[t] = f32x16{};
  float m_run = -__builtin_inff();   // reference max, log2 units (same in lanes l and l ^ 32)
  float l_run = 0.f;                 // running sum over this lane's keys

  for (int w0 = 0; w0 < nblk; w0 += kPfWindow) {
    const int w1 = min(nblk, w0 + kPfWindow);
    barrier();   // the ring is free: every wave is done with the last window's units
    // The window's metadata stays in registers: lane i holds the table entry
    // of block w0 + i, and a 64-bit mask holds the BASE tags, so a DMA issue
    // reads its block id with one lane read and no LDS round trip.
    int bt_lane = 0;
    bool base_lane = false;
    if (w0 + lane < w1) {
      const int bt = btrow[w0 + lane];
      bt_lane = (unsigned)bt < (unsigned)a.num_blocks ? bt : 0;   // never leave the pool
      if constexpr (ELASTIC)
        base_lane = use_tags ? tagrow[w0 + lane] != 0 : (w0 + lane >= base_lo && w0 + lane < base_hi);
    }
    const uint64_t base_mask = __builtin_amdgcn_ballot_w64(base_lane);   // bit i: block w0 + i is BASE

    auto is_base = [&](int blk) -> bool {
      if constexpr (!ELASTIC) return false;
      else return ((base_mask >> (blk - w0)) & 1) != 0;
    };
    int ib = w0, issued = 0, consumed = 0;
    auto issue = [&]() {
      const bool base = is_base(ib);
      const char* src = pool + (size_t)(uint32_t)__builtin_amdgcn_readlane(bt_lane, ib - w0) * block_bytes;
      const uint32_t dst = lds_wave + (uint32_t)(issued & (kPfRing - 1)) * kSlotBytes;
      if constexpr (F8) {
        if (base) {
          // both members' nibbles (2 KiB per plane) to the staging area: this
          // wave moves 512 B of K and of V with half its lanes
          const uint32_t nd = nib_wave + (uint32_t)(issued & (kPfRing - 1)) * kTileBytes;
          if (lane < 32) {
            const char* ns = src + 512 * wave + 16 * lane;
            __builtin_amdgcn_global_load_lds(static_cast<const void*>(ns), (lds_ptr)(size_t)nd, 16, 0, 0);
            __builtin_amdgcn_global_load_lds(static_cast<const void*>(ns + v_off), (lds_ptr)(size_t)(nd + kTileBytes / 2),
                                             16, 0, 0);
          }
          ib += 2;
        } else {
          // member m of a TARGET pair from its own block; a lone last block
          // stands in for the missing member 1 (whose keys are masked)
          const bool pair = ib + 1 < w1;
          const int b1 = pair ? __builtin_amdgcn_readlane(bt_lane, ib + 1 - w0) : 0;
          const char* srcm = (wave >> 1) && pair ? pool + (size_t)(uint32_t)b1 * block_bytes : src;
          __builtin_amdgcn_global_load_lds(static_cast<const void*>(srcm + dma_member), (lds_ptr)(size_t)dst, 16, 0, 0);
          __builtin_amdgcn_global_load_lds(static_cast<const void*>(srcm + v_off + dma_member),
                                           (lds_ptr)(size_t)(dst + kTileBytes), 16, 0, 0);
          ib += pair ? 2 : 1;
        }
      } else {
        const uint32_t off = base ? dma.base[0] : dma_tgt;
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + off), (lds_ptr)(size_t)dst, 16, 0, 0);
        __builtin_amdgcn_global_load_lds(static_cast<const void*>(src + v_off + off),
                                         (lds_ptr)(size_t)(dst + kTileBytes), 16, 0, 0);
        ib += base ? 2 : 1;
      }
      ++issued;
    };
#pragma unroll
    for (int k = 0; k < kPfRing - 1; ++k)
      if (ib < w1) issue();

    for (int cb = w0; cb < w1;) {
      // the unit: a BASE pair (one slot), two TARGET blocks, or a lone block
      const bool base = is_base(cb);
      const bool two = !F8 && !base && cb + 1 < w1;   // 8-bit units take one slot each
      const int nslots = two ? 2 : 1;
      while (issued < consumed + nslots) issue();   // (the ring normally runs ahead)
      wait_slots(issued - consumed - nslots);
      barrier();   // every wave's quarters have landed; the slots of the last unit are free
      while (ib < w1 && issued - consumed < kPfRing) issue();

      const char* sa = ring[consumed & (kPfRing - 1)];
      const char* sbk = ring[(consumed + (two ? 1 : 0)) & (kPfRing - 1)];
      const int key0 = cb * kPage;
      const bool full = base || cb + 1 < w1;   // two blocks in the unit (else the lone last one)
      const int nkeys = full ? 32 : 16;
      if constexpr (F8) {
        if (base) {
          // widen the staged nibbles: each lane makes one 16-byte chunk of K
          // and one of V (member m, row t, chunk q at position q ^ tau(t))
          const int p = lane + 64 * wave;
          const int m = p >> 7, t = (p >> 3) & 15, qc = p & 7;
          const char* ns = nib[consumed & (kPfRing - 1)] + m * (kTileBytes / 4) + t * (kHeadDim / 2) + 8 * qc;
          char* bd = ring[consumed & (kPfRing - 1)] + m * (kTileBytes / 2) + t * kHeadDim + 16 * (qc ^ tau(t));
#pragma unroll
          for (int plane = 0; plane < 2; ++plane) {
            const u32x2 x = *reinterpret_cast<const u32x2*>(ns + plane * (kTileBytes / 2));
            const u32x2 lo = widen_nibbles(x.x), hi = widen_nibbles(x.y);
            *reinterpret_cast<u32x4*>(bd + plane * kTileBytes) = u32x4{lo.x, lo.y, hi.x, hi.y};
          }
          barrier();   // the widened tiles are visible to every wave
        }
      }

      // The block kind only changes how the K and V operands are fetched:
      // each fetch phase branches once on it (not once per step), so a
      // phase's LDS reads are all in flight together, while the products
      // and the accumulators stay in code common to both kinds.
      auto unit = [&](auto masked) {
        constexpr bool kMasked = decltype(masked)::value;
        // ---- S^T = K Q^T ----
        u32x4 kop[8];
        if (F8 || (ELASTIC && base)) {
#pragma unroll
          for (int k = 0; k < 8; ++k)
            kop[k] = expand_base8(*reinterpret_cast<const u32x2*>(sa + (off_kb ^ (16 * k))));
        } else {
          const char* sk = n < 16 ? sa : sbk;   // the lane's key row is in its member's slot
#pragma unroll
          for (int k = 0; k < 8; ++k) kop[k] = *reinterpret_cast<const u32x4*>(sk + (off_kt ^ (32 * k)));
        }
        f32x16 sc = f32x16{};
#pragma unroll
        for (int k = 0; k < 8; ++k) sc = Mma32<T>::mma(kop[k], qop[k], sc);

        // V^T operands of key step ks (16 keys); step 0 is fetched before the
        // softmax, so its LDS reads overlap the wait for the S^T products
        struct VOps {
          u32x4 t[4];
        };
        auto fetch_v = [&](int ks) -> VOps {
          VOps r;
          if (F8 || (ELASTIC && base)) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const i32x2v raw =
                  __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2)(sa + ks * (kTileBytes / 2) + (off_vb ^ (32 * t))));
              r.t[t] = expand_base8(u32x2{(uint32_t)raw[0], (uint32_t)raw[1]});
              if (F8 && kMasked) {   // 8-bit TARGET keys at or past the sequence end: zero V
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  const int key = 16 * ks + 8 * (e >> 2) + 4 * h + (e & 3);
                  if (key0 + key >= len) r.t[t][e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
                }
              }
            }
          } else {
            const char* sl = ks == 0 ? sa : sbk;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              uint32_t w[4];
#pragma unroll
              for (int half = 0; half < 2; ++half) {
                const u32x2 pr = __builtin_bit_cast(
                    u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4)(sl + (off_vt[half] ^ (64 * t)))));
                w[2 * half] = pr.x;
                w[2 * half + 1] = pr.y;
              }
              if (kMasked) {   // keys at or past the sequence end: zero V (their slots hold anything)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                  const int key = 16 * ks + 8 * (e >> 2) + 4 * h + (e & 3);
                  if (key0 + key >= len) w[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
                }
              }
              r.t[t] = u32x4{w[0], w[1], w[2], w[3]};
            }
          }
          return r;
        };
        const VOps v0 = fetch_v(0);

        // ---- online softmax over this lane's 16 keys (+ lane ^ 32) ----
        // Scores enter the softmax as s * c in log2 units.  Interior units fold
        // c into the max and the exponent; masked units scale first and then
        // set masked keys to -inf, so that a zero scale never multiplies an
        // infinity (0 * -inf is NaN).
        const float c = kMasked ? 1.0f : c_scale;
        if constexpr (kMasked) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = 8 * (r >> 2) + 4 * h + (r & 3);
            sc[r] = (key >= nkeys || key0 + key >= lim) ? -__builtin_inff() : sc[r] * c_scale;
          }
        }
        const float m0 = max3(sc[0], sc[1], sc[2]), m1 = max3(sc[3], sc[4], sc[5]);
        const float m2 = max3(sc[6], sc[7], sc[8]), m3 = max3(sc[9], sc[10], sc[11]);
        const float m4 = max3(sc[12], sc[13], sc[14]);
        float mx = max3(max3(m0, m1, m2), max3(m3, m4, sc[15]), m0);
        {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
          mx = max3(__uint_as_float(sw[0]), __uint_as_float(sw[1]), __uint_as_float(sw[1])) * c;
        }
        if (__builtin_amdgcn_ballot_w64(mx > m_run + 8.0f)) {
          const float m_new = fmaxf(m_run, mx);
          const float alpha = fast_exp2(m_run - m_new);
          l_run *= alpha;
#pragma unroll
          for (int t = 0; t < 4; ++t) scale_in_place(o[t], alpha);
          m_run = m_new;
        }
        // P = exp2(s c - m); its 16-bit head by truncation, the remainder
        // p - head rounded to 16 bits
        u32x4 phi[2], plo[2];
        float lsum[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          float p[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) p[i] = fast_exp2(__builtin_fmaf(sc[8 * ks + i], c, -m_run));
          lsum[ks] = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
          uint32_t wh[4], wl[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) split_p<T>(p[2 * u], p[2 * u + 1], wh[u], wl[u]);
          phi[ks] = u32x4{wh[0], wh[1], wh[2], wh[3]};
          plo[ks] = u32x4{wl[0], wl[1], wl[2], wl[3]};
        }
        l_run += lsum[0] + lsum[1];

        // ---- O^T += V^T P^T (16-bit head and remainder of P) ----
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          if (kMasked && ks == 1 && nkeys < 32) break;
          const VOps v = ks == 0 ? v0 : fetch_v(1);
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            o[t] = Mma32<T>::mma(v.t[t], phi[ks], o[t]);
            o[t] = Mma32<T>::mma(v.t[t], plo[ks], o[t]);
          }
        }
      };
      if (key0 + nkeys > lim_wave || nkeys < 32) unit(std::true_type{});
      else unit(std::false_type{});
      consumed += nslots;
      cb += full ? 2 : 1;
    }
  }

  // ---- output: this lane holds dims 32t + 8u + 4h .. + 3 of its column ----
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_run), __float_as_uint(l_run), false, false);
  const float l_tot = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  if (col_ok) {
    const float inv = 1.0f / l_tot;
    const size_t row = ((size_t)(q0 + tq) * a.num_q_heads + (size_t)kvh * G + head) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const size_t idx = row + 32 * t + 8 * u + 4 * h;
        store_pair<T>(a.out, idx, o[t][4 * u] * inv, o[t][4 * u + 1] * inv, a.out_fp32);
        store_pair<T>(a.out, idx + 2, o[t][4 * u + 2] * inv, o[t][4 * u + 3] * inv, a.out_fp32);
      }
  }
}

template <typename T, int G, bool F8>
hipError_t launch_typed(const PrefillArgs& a, bool elastic, hipStream_t st) {
  constexpr int kTileTok = kPfWaves * kPfCols / G;
  dim3 grid((a.max_q_len + kTileTok - 1) / kTileTok, a.num_kv_heads, a.batch);
  if (elastic) hipLaunchKernelGGL((prefill_kernel<T, G, true, F8>), grid, dim3(64 * kPfWaves), 0, st, a);
  else hipLaunchKernelGGL((prefill_kernel<T, G, false, F8>), grid, dim3(64 * kPfWaves), 0, st, a);
  return hipGetLastError();
}

template <typename T, bool F8>
hipError_t launch_group(const PrefillArgs& a, int group, bool elastic, hipStream_t st) {
  switch (group) {
    case 1: return launch_typed<T, 1, F8>(a, elastic, st);
    case 2: return launch_typed<T, 2, F8>(a, elastic, st);
    case 4: return launch_typed<T, 4, F8>(a, elastic, st);
    case 8: return launch_typed<T, 8, F8>(a, elastic, st);
    case 16: return launch_typed<T, 16, F8>(a, elastic, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, int dtype, int group, bool elastic, hipStream_t st) {
  if (a.batch == 0 || a.max_q_len == 0) return hipSuccess;
  if (dtype == 3) return launch_group<Fp16, true>(a, group, elastic, st);   // 8-bit pool, FP16 queries
  return dtype == 0 ? launch_group<Bf16, false>(a, group, elastic, st) : launch_group<Fp16, false>(a, group, elastic, st);
}

}  // namespace ekv
