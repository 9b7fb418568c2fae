// Fidelity transitions (paper §3.1; §3.4 "Transition protocols"; App. B.2)
// and the TARGET append of new KV (§3.2).
//
// Demotion packs the high bytes of a TARGET pair into member 0's block and
// emits the low bytes; refinement rebuilds both members' words from the
// packed high bytes and the stored low bytes.  In the packed layout every
// (plane, head) 4 KiB tile of the kept block holds exactly the bytes of the
// same (plane, head) tiles of the two members, so one wave owns one tile
// end to end: it reads everything it needs into registers, waits for all
// its loads to land, then overwrites the tile.  No two waves touch the
// same bytes, which is what makes the in-place rewrite race-free.
//
// Block-table and tag updates run in a second, tiny kernel after the data
// kernel on the same stream, so no data wave can observe a half-updated
// table.
//
// A staged refinement finds a pair's refinement bytes in its new block Q,
// where an asynchronous host-to-device copy put them while the pair stayed
// BASE (App. B.2): every wave reads its whole P and Q tiles before writing
// either, so rebuilding Q over its own staged bytes is still tile-local.
//
// The staging copy of asynchronous promotion moves each pair's backed-up
// refinement bytes into its new block.  Its sources are usually pinned host
// memory mapped for the device, so the copy is a kernel that reads over the
// host link: one launch keeps thousands of 16-byte reads in flight, where
// one DMA copy per block pays a fixed cost per block.
//
// A multi-layer call transforms the same pairs in every layer's pool in one
// launch (grid z = layer): the layers share one block table, as the layers
// of a paged serving runtime do, so the table is read by every layer's
// waves and committed once.
#include "common.h"
#include "launch.h"

namespace ekv {
namespace {

// 16-bit words -> their high / low bytes (4 words per u32x2).
__device__ __forceinline__ uint32_t hi_bytes(u32x2 w) { return perm(w.y, w.x, 0x07050301u); }
__device__ __forceinline__ uint32_t lo_bytes(u32x2 w) { return perm(w.y, w.x, 0x06040200u); }
// (hi byte, lo byte) pairs -> 16-bit words: 4 words from one dword of each.
__device__ __forceinline__ u32x2 join_words(uint32_t hi, uint32_t lo) {
  return u32x2{perm(hi, lo, 0x05010400u), perm(hi, lo, 0x07030602u)};
}

__device__ __forceinline__ void wait_all_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The pool of this workgroup's layer (grid z) and its refinement bytes of pair i.
__device__ __forceinline__ uint16_t* layer_pool(const TransitionArgs& a) {
  return a.layers ? reinterpret_cast<uint16_t*>(a.layers[blockIdx.z]) : a.pool;
}
__device__ __forceinline__ size_t lo_offset(const TransitionArgs& a, int i, size_t block_words) {
  return ((size_t)i * a.num_layers + blockIdx.z) * (2 * block_words);
}

// A list entry that points outside the arrays the call was given (a
// sequence beyond the table, a pair beyond its row, a block beyond the
// pool) is skipped by every kernel, so an invalid list cannot make a call
// touch memory outside them.  Lists are validated on the host mirrors
// (ekv_check_transition); for invalid lists the results are undefined.
__device__ __forceinline__ bool pair_ok(const TransitionArgs& a, int s, int j) {
  return (unsigned)s < (unsigned)a.batch && j >= 0 && 2 * j + 1 < a.max_blocks;
}
__device__ __forceinline__ bool block_ok(const TransitionArgs& a, int b) { return (unsigned)b < (unsigned)a.num_blocks; }
// the pair's two table entries, or false
__device__ __forceinline__ bool pair_blocks(const TransitionArgs& a, int s, int j, int& b0, int& b1) {
  if (!pair_ok(a, s, j)) return false;
  const int32_t* row = a.bt + (size_t)s * a.max_blocks;
  b0 = row[2 * j];
  b1 = row[2 * j + 1];
  return block_ok(a, b0) && block_ok(a, b1);
}

__global__ __launch_bounds__(64) void demote_kernel(TransitionArgs a) {
  const int tile = blockIdx.x;   // plane * Hkv + head
  const int i = blockIdx.y;
  const int lane = threadIdx.x;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int b0 = 0, b1 = 0;
  if (!pair_blocks(a, s, j, b0, b1)) return;
  const size_t block_words = (size_t)2 * a.num_kv_heads * kTileWords;
  uint16_t* pool = layer_pool(a);
  uint16_t* t0 = pool + (size_t)b0 * block_words + (size_t)tile * kTileWords;
  const uint16_t* t1 = pool + (size_t)b1 * block_words + (size_t)tile * kTileWords;

  u32x4 w0[4], w1[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    w0[r] = *reinterpret_cast<const u32x4*>(t0 + 8 * lane + 512 * r);
    w1[r] = *reinterpret_cast<const u32x4*>(t1 + 8 * lane + 512 * r);
  }
  wait_all_loads();
  uint8_t* packed = reinterpret_cast<uint8_t*>(t0);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int off = 8 * lane + 512 * r;   // word index within the tile = byte index within a member
    *reinterpret_cast<u32x2*>(packed + off) = u32x2{hi_bytes(w0[r].xy), hi_bytes(w0[r].zw)};
    *reinterpret_cast<u32x2*>(packed + kTileBytes / 2 + off) = u32x2{hi_bytes(w1[r].xy), hi_bytes(w1[r].zw)};
  }
  if (a.lo) {
    uint8_t* lo = a.lo + lo_offset(a, i, block_words) + (size_t)tile * kTileBytes;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int off = 8 * lane + 512 * r;
      *reinterpret_cast<u32x2*>(lo + off) = u32x2{lo_bytes(w0[r].xy), lo_bytes(w0[r].zw)};
      *reinterpret_cast<u32x2*>(lo + kTileBytes / 2 + off) = u32x2{lo_bytes(w1[r].xy), lo_bytes(w1[r].zw)};
    }
  }
}

__global__ __launch_bounds__(256) void demote_commit_kernel(TransitionArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int b0 = 0, b1 = 0;
  if (!pair_blocks(a, s, j, b0, b1)) {
    a.freed[i] = -1;   // skipped entry: nothing was freed
    return;
  }
  int32_t* row = a.bt + (size_t)s * a.max_blocks;
  uint8_t* tg = a.tags + (size_t)s * a.max_blocks;
  a.freed[i] = b1;
  row[2 * j + 1] = b0;
  tg[2 * j] = 1;
  tg[2 * j + 1] = 1;
}

__global__ __launch_bounds__(64) void refine_kernel(TransitionArgs a) {
  const int tile = blockIdx.x;
  const int i = blockIdx.y;
  const int lane = threadIdx.x;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int bp = 0, b1 = 0;
  const int bq = a.new_blocks[i];
  if (!pair_blocks(a, s, j, bp, b1) || !block_ok(a, bq)) return;
  const size_t block_words = (size_t)2 * a.num_kv_heads * kTileWords;
  uint16_t* pool = layer_pool(a);
  uint16_t* tp = pool + (size_t)bp * block_words + (size_t)tile * kTileWords;
  uint16_t* tq = pool + (size_t)bq * block_words + (size_t)tile * kTileWords;
  const uint8_t* packed = reinterpret_cast<const uint8_t*>(tp);
  // staged: the refinement bytes were copied into Q itself; its (plane, head)
  // tile holds exactly the bytes this wave rebuilds that tile from
  const uint8_t* lo = a.staged ? reinterpret_cast<const uint8_t*>(tq)
                               : a.lo + lo_offset(a, i, block_words) + (size_t)tile * kTileBytes;

  u32x2 h0[4], h1[4], l0[4], l1[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int off = 8 * lane + 512 * r;
    h0[r] = *reinterpret_cast<const u32x2*>(packed + off);
    h1[r] = *reinterpret_cast<const u32x2*>(packed + kTileBytes / 2 + off);
    l0[r] = *reinterpret_cast<const u32x2*>(lo + off);
    l1[r] = *reinterpret_cast<const u32x2*>(lo + kTileBytes / 2 + off);
  }
  wait_all_loads();
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int off = 8 * lane + 512 * r;
    const u32x2 a0 = join_words(h0[r].x, l0[r].x), b0 = join_words(h0[r].y, l0[r].y);
    const u32x2 a1 = join_words(h1[r].x, l1[r].x), b1 = join_words(h1[r].y, l1[r].y);
    *reinterpret_cast<u32x4*>(tp + off) = u32x4{a0.x, a0.y, b0.x, b0.y};
    *reinterpret_cast<u32x4*>(tq + off) = u32x4{a1.x, a1.y, b1.x, b1.y};
  }
}

// ---- 8-bit TARGET / 4-bit BASE ---------------------------------------------
// A (plane, head) tile is 2 KiB (16 rows of 128 bytes); a packed tile holds
// [member 0 | member 1] nibble rows of 64 bytes, element e of a row in byte
// e / 2 (low nibble when e is even).  Lane L owns the 32 bytes [32L, 32L+32)
// of each member's TARGET tile, i.e. the 16 packed bytes [16L, 16L+16) of
// that member's half.
constexpr int kTile8 = kPage * kHeadDim;   // 2 KiB

// Four bytes (one nibble of each, in the low nibble) -> bytes 0 and 2 of the
// result hold nibbles (0 | 1 << 4) and (2 | 3 << 4).
__device__ __forceinline__ uint32_t pair_nibbles(uint32_t t) { return t | (t >> 4); }

// 32 TARGET bytes -> 16 bytes of their high (hi = true) or low nibbles.
__device__ __forceinline__ u32x4 pack_nibbles(const u32x4 (&x)[2], bool hi) {
  uint32_t w[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const uint32_t in = x[q >> 2][q & 3];
    w[q] = pair_nibbles(hi ? (in >> 4) & 0x0F0F0F0Fu : in & 0x0F0F0F0Fu);
  }
  return u32x4{perm(w[1], w[0], 0x06040200u), perm(w[3], w[2], 0x06040200u), perm(w[5], w[4], 0x06040200u),
               perm(w[7], w[6], 0x06040200u)};
}

// 4 bytes of high nibbles + 4 bytes of low nibbles -> 8 TARGET bytes.
__device__ __forceinline__ u32x2 join_nibbles(uint32_t h, uint32_t l) {
  const uint32_t even = ((h & 0x0F0F0F0Fu) << 4) | (l & 0x0F0F0F0Fu);
  const uint32_t odd = (h & 0xF0F0F0F0u) | ((l >> 4) & 0x0F0F0F0Fu);
  return u32x2{perm(odd, even, 0x05010400u), perm(odd, even, 0x07030602u)};
}

__device__ __forceinline__ uint8_t* layer_pool8(const TransitionArgs& a) {
  return reinterpret_cast<uint8_t*>(layer_pool(a));
}

__global__ __launch_bounds__(64) void demote8_kernel(TransitionArgs a) {
  const int tile = blockIdx.x;
  const int i = blockIdx.y;
  const int lane = threadIdx.x;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int b0 = 0, b1 = 0;
  if (!pair_blocks(a, s, j, b0, b1)) return;
  const size_t block_bytes = (size_t)2 * a.num_kv_heads * kTile8;
  uint8_t* pool = layer_pool8(a);
  uint8_t* t0 = pool + (size_t)b0 * block_bytes + (size_t)tile * kTile8;
  const uint8_t* t1 = pool + (size_t)b1 * block_bytes + (size_t)tile * kTile8;
  u32x4 x0[2], x1[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    x0[r] = *reinterpret_cast<const u32x4*>(t0 + 32 * lane + 16 * r);
    x1[r] = *reinterpret_cast<const u32x4*>(t1 + 32 * lane + 16 * r);
  }
  wait_all_loads();
  *reinterpret_cast<u32x4*>(t0 + 16 * lane) = pack_nibbles(x0, true);
  *reinterpret_cast<u32x4*>(t0 + kTile8 / 2 + 16 * lane) = pack_nibbles(x1, true);
  if (a.lo) {
    uint8_t* lo = a.lo + ((size_t)i * a.num_layers + blockIdx.z) * block_bytes + (size_t)tile * kTile8;
    *reinterpret_cast<u32x4*>(lo + 16 * lane) = pack_nibbles(x0, false);
    *reinterpret_cast<u32x4*>(lo + kTile8 / 2 + 16 * lane) = pack_nibbles(x1, false);
  }
}

__global__ __launch_bounds__(64) void refine8_kernel(TransitionArgs a) {
  const int tile = blockIdx.x;
  const int i = blockIdx.y;
  const int lane = threadIdx.x;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int bp = 0, b1 = 0;
  const int bq = a.new_blocks[i];
  if (!pair_blocks(a, s, j, bp, b1) || !block_ok(a, bq)) return;
  const size_t block_bytes = (size_t)2 * a.num_kv_heads * kTile8;
  uint8_t* pool = layer_pool8(a);
  uint8_t* tp = pool + (size_t)bp * block_bytes + (size_t)tile * kTile8;
  uint8_t* tq = pool + (size_t)bq * block_bytes + (size_t)tile * kTile8;
  const uint8_t* lo = a.staged ? tq : a.lo + ((size_t)i * a.num_layers + blockIdx.z) * block_bytes + (size_t)tile * kTile8;
  u32x4 h[2], l[2];
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    h[m] = *reinterpret_cast<const u32x4*>(tp + m * (kTile8 / 2) + 16 * lane);
    l[m] = *reinterpret_cast<const u32x4*>(lo + m * (kTile8 / 2) + 16 * lane);
  }
  wait_all_loads();
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    uint8_t* dst = m ? tq : tp;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const u32x2 a0 = join_nibbles(h[m][2 * r], l[m][2 * r]);
      const u32x2 a1 = join_nibbles(h[m][2 * r + 1], l[m][2 * r + 1]);
      *reinterpret_cast<u32x4*>(dst + 32 * lane + 16 * r) = u32x4{a0.x, a0.y, a1.x, a1.y};
    }
  }
}

__global__ __launch_bounds__(256) void refine_commit_kernel(TransitionArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  int bp = 0, b1 = 0;
  if (!pair_blocks(a, s, j, bp, b1) || !block_ok(a, a.new_blocks[i])) return;
  a.bt[(size_t)s * a.max_blocks + 2 * j + 1] = a.new_blocks[i];
  uint8_t* tg = a.tags + (size_t)s * a.max_blocks;
  tg[2 * j] = 0;
  tg[2 * j + 1] = 0;
}

// One wave per new token: 2*Hkv rows of 256 B (16 lanes per row), or of
// 128 B for 1-byte elements (8 lanes per row).
__global__ __launch_bounds__(64) void append8_kernel(AppendArgs a) {
  const int i = blockIdx.x;
  const int lane = threadIdx.x;
  const int slot = a.slots[i];
  if (slot < 0 || slot / kPage >= a.num_blocks) return;   // outside the pool: skipped
  const int blk = slot / kPage, off = slot % kPage;
  const int hkv = a.num_kv_heads;
  const size_t block_bytes = (size_t)2 * hkv * kTile8;
  const int c = lane & 7;
  const uint8_t* k = reinterpret_cast<const uint8_t*>(a.k);
  const uint8_t* v = reinterpret_cast<const uint8_t*>(a.v);
  uint8_t* pool = reinterpret_cast<uint8_t*>(a.pool);
  for (int r = lane >> 3; r < 2 * hkv; r += 8) {
    const int plane = r / hkv, h = r % hkv;
    const uint8_t* src = (plane ? v : k) + ((size_t)i * hkv + h) * kHeadDim + 16 * c;
    uint8_t* dst = pool + (size_t)blk * block_bytes + (size_t)r * kTile8 + off * kHeadDim + 16 * c;
    *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
  }
}

__global__ __launch_bounds__(64) void append_kernel(AppendArgs a) {
  const int i = blockIdx.x;
  const int lane = threadIdx.x;
  const int slot = a.slots[i];
  if (slot < 0 || slot / kPage >= a.num_blocks) return;   // outside the pool: skipped
  const int blk = slot / kPage, off = slot % kPage;
  const int hkv = a.num_kv_heads;
  const size_t block_words = (size_t)2 * hkv * kTileWords;
  const int c = lane & 15;
  for (int r = lane >> 4; r < 2 * hkv; r += 4) {
    const int plane = r / hkv, h = r % hkv;
    const uint16_t* src = (plane ? a.v : a.k) + ((size_t)i * hkv + h) * kHeadDim + 8 * c;
    uint16_t* dst = a.pool + (size_t)blk * block_words + (size_t)r * kTileWords + off * kHeadDim + 8 * c;
    *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
  }
}

// One 4 KiB piece of one block per workgroup, 16 bytes a lane.
__global__ __launch_bounds__(256) void stage_kernel(StageArgs a) {
  const int i = blockIdx.y;
  const size_t off = (size_t)blockIdx.x * 4096 + 16 * threadIdx.x;
  const u32x4 v = *reinterpret_cast<const u32x4*>(a.src[i] + off);
  *reinterpret_cast<u32x4*>(a.pool + (size_t)a.dst[i] * a.block_bytes + off) = v;
}

}  // namespace

hipError_t launch_stage(const StageArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(stage_kernel, dim3((unsigned)(a.block_bytes / 4096), a.n), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_demote(const TransitionArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(a.elem8 ? demote8_kernel : demote_kernel, dim3(2 * a.num_kv_heads, a.n, a.num_layers),
                     dim3(64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(demote_commit_kernel, dim3((a.n + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_refine(const TransitionArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(a.elem8 ? refine8_kernel : refine_kernel, dim3(2 * a.num_kv_heads, a.n, a.num_layers),
                     dim3(64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(refine_commit_kernel, dim3((a.n + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(a.elem8 ? append8_kernel : append_kernel, dim3(a.n), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace ekv
