// C ABI of libekv: argument checks, dispatch-metadata lowering, split-KV
// planning, and kernel dispatch.  Declarations and contracts: include/ekv.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "ekv.h"
#include "common.h"
#include "host_status.h"
#include "launch.h"

namespace {

thread_local char g_last_error[512];

}  // namespace

namespace ekv {

ekv_status fail(ekv_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return s;
}

}  // namespace ekv

namespace {

using ekv::fail;

ekv_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return EKV_OK;
  return fail(EKV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool supported_group(int g) { return g == 1 || g == 2 || g == 4 || g == 8 || g == 16; }

ekv_status check_pool(const ekv_pool* p) {
  if (!p) return fail(EKV_ERR_INVALID, "pool is NULL");
  if (!p->kv) return fail(EKV_ERR_INVALID, "pool->kv is NULL");
  if (p->num_blocks <= 0 || p->num_kv_heads <= 0)
    return fail(EKV_ERR_INVALID, "pool sizes must be positive");
  if (p->head_dim != ekv::kHeadDim || p->page_size != ekv::kPage)
    return fail(EKV_ERR_UNSUPPORTED, "only head_dim 128 and page_size 16 are supported");
  if (p->dtype != EKV_DTYPE_BF16 && p->dtype != EKV_DTYPE_FP16 && p->dtype != EKV_DTYPE_E5M2)
    return fail(EKV_ERR_UNSUPPORTED, "pool dtype must be bf16, fp16 or e5m2");
  if (p->num_kv_heads > 64) return fail(EKV_ERR_UNSUPPORTED, "at most 64 KV heads");
  return EKV_OK;
}

ekv_status check_attention_batch(const ekv_pool* p, const ekv_batch* b, int* group) {
  if (!b) return fail(EKV_ERR_INVALID, "batch is NULL");
  if (b->batch < 0 || b->max_blocks <= 0 || b->num_q_heads <= 0)
    return fail(EKV_ERR_INVALID, "batch sizes must be positive");
  if (b->num_q_heads % p->num_kv_heads)
    return fail(EKV_ERR_INVALID, "num_q_heads must be a multiple of num_kv_heads");
  *group = b->num_q_heads / p->num_kv_heads;
  if (!supported_group(*group)) return fail(EKV_ERR_UNSUPPORTED, "group size %d not supported", *group);
  if (b->batch > 0 && (!b->seq_lens || !b->block_table))
    return fail(EKV_ERR_INVALID, "seq_lens and block_table are required");
  if (b->mode < EKV_MODE_NATIVE || b->mode > EKV_MODE_GENERAL)
    return fail(EKV_ERR_INVALID, "unknown mode %d", b->mode);
  if (b->mode == EKV_MODE_STRUCTURED && !b->boundaries && !b->tags)
    return fail(EKV_ERR_INVALID, "structured mode needs boundaries (or tags)");
  if (b->mode == EKV_MODE_GENERAL && !b->tags)
    return fail(EKV_ERR_INVALID, "general mode needs the tag table");
  if ((long long)b->max_seq_len > (long long)b->max_blocks * ekv::kPage || b->max_seq_len < 0)
    return fail(EKV_ERR_INVALID, "max_seq_len exceeds max_blocks * page_size");
  return EKV_OK;
}

int max_seq_blocks(const ekv_batch* b) {
  const int len = b->max_seq_len > 0 ? b->max_seq_len : b->max_blocks * ekv::kPage;
  return (len + ekv::kPage - 1) / ekv::kPage;
}

// Fewest pairs (32 tokens) one workgroup streams; EKV_MIN_CHUNK overrides.
int plan_min_chunk() {
  if (const char* env = getenv("EKV_MIN_CHUNK")) {
    const int v = atoi(env);
    if (v > 0) return v;
  }
  return 8;
}

// LDS ring depth of the decode kernel: the deepest ring that still lets 4
// workgroups (one per SIMD) share a CU's 160 KiB with their window buffers.
// 8-bit pools holding BASE pairs: per-pair work outweighs the halved bytes,
// so twice the waves per SIMD (a shallower ring) pay more than depth.
int decode_slots(const ekv_pool* p, int group, bool elastic) {
  int slots = group <= 4 ? 4 : (group == 8 ? 3 : 2);
  if (p->dtype == EKV_DTYPE_E5M2 && elastic) slots = 2;
  if (const char* env = getenv("EKV_DECODE_SLOTS")) slots = std::max(2, std::min(4, atoi(env)));
  return slots;
}

// Workspace: [merge counters u32, 2 kMaxDecodeGrid | (m, l) f32 | o f32
// rows], 256-B aligned parts; the last two hold two slots per workgroup of
// the launch (G rows a slot), the counters two per possible workgroup.
// The launch grid is the kernel's resident workgroups on the device, or
// fewer for small work, and never more than kMaxDecodeGrid.  The size a
// caller allocates (exact = false) bounds the grid by the work and that cap
// only, so it needs no device and serves every mode of a batch shape; the
// size a call needs (exact = true) uses the device's own grid, the larger
// of the native and the elastic kernel's.
struct DecodePlan {
  int min_chunk, grid;      // grid of the call's own mode (exact plans)
  long long pairs_max;
  size_t ml_offset, o_offset, total;
};

ekv_status plan_decode(const ekv_pool* p, const ekv_batch* b, int group, bool exact, DecodePlan* d) {
  const int nblk = std::max(1, max_seq_blocks(b));
  const int np_max = (nblk + 1) / 2;
  d->min_chunk = plan_min_chunk();
  d->pairs_max = (long long)b->batch * p->num_kv_heads * np_max;
  if (d->pairs_max >= (1LL << 30)) return fail(EKV_ERR_UNSUPPORTED, "batch too large for one decode call");
  const long long wanted = (d->pairs_max + d->min_chunk - 1) / d->min_chunk;
  int grids[2] = {0, 0};
  for (int elastic = 0; elastic < 2; ++elastic) {
    if (!exact) {
      grids[elastic] = (int)std::max<long long>(1, std::min<long long>(wanted, ekv::kMaxDecodeGrid));
      continue;
    }
    ekv::DecodeArgs a{};
    a.pairs_max = d->pairs_max;
    a.min_chunk = d->min_chunk;
    a.slots = decode_slots(p, group, elastic != 0);
    const hipError_t e = ekv::decode_grid(a, p->dtype, group, elastic != 0, &grids[elastic]);
    if (e != hipSuccess) return hip_status(e, "decode grid");
  }
  d->grid = grids[b->mode != EKV_MODE_NATIVE ? 1 : 0];
  const size_t slots = 2 * (size_t)std::max(grids[0], grids[1]);
  auto align = [](size_t x) { return (x + 255) & ~(size_t)255; };
  // The counters keep one place whatever the grid: a workspace reused by
  // calls whose grids differ (other batch sizes) never finds partial rows
  // of an earlier call where a later call expects zero counters.
  d->ml_offset = align(2 * (size_t)ekv::kMaxDecodeGrid * sizeof(uint32_t));
  d->o_offset = align(d->ml_offset + slots * group * 2 * sizeof(float));
  d->total = d->o_offset + slots * group * ekv::kHeadDim * sizeof(float);
  return EKV_OK;
}

// The no-allocation decode's scratch: one array per device (each GPU the
// library runs on holds its own copy until the process ends).  Host code
// never uses its name as an address: scratch_address() looks up the
// device's address of the array once per device, with that device current.
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kScratchDevices = 64;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

ekv_status scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[kScratchDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hip_status(hipGetLastError(), "hipGetDevice");
  if (dev < 0 || dev >= kScratchDevices) return fail(EKV_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kScratchDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    addr[dev] = ptr;
  }
  *out = addr[dev];
  return EKV_OK;
}

float log2e_scale(float scale) { return scale * 1.4426950408889634f; }

// ---- device-side validation and the EKV_DEBUG mode ------------------------

const char* violation_name(int k) {
  static const char* const names[EKV_VIOL_COUNT] = {
      "sequence length out of range", "table entry outside the pool", "tag value",
      "pair with mixed tags", "BASE pair that is not two full blocks", "BASE pair with two table entries",
      "mode or boundaries disagree with the tags", "list pair out of range", "list pair in the wrong state",
      "list pair not two full blocks", "list pair listed twice", "new block out of range, repeated or in use"};
  return k >= 0 && k < EKV_VIOL_COUNT ? names[k] : "unknown";
}

bool debug_mode() {
  const char* e = getenv("EKV_DEBUG");
  return e && e[0] && strcmp(e, "0") != 0;
}

ekv_status check_validate_batch(const ekv_pool* pool, const ekv_batch* batch, int32_t* report) {
  ekv_status st = check_pool(pool);
  if (st != EKV_OK) return st;
  int group = 0;
  if ((st = check_attention_batch(pool, batch, &group)) != EKV_OK) return st;
  if (!report) return fail(EKV_ERR_INVALID, "report is required");
  if ((long long)batch->batch * batch->max_blocks >= (1LL << 31))
    return fail(EKV_ERR_UNSUPPORTED, "batch * max_blocks must be below 2^31");
  return EKV_OK;
}

hipError_t enqueue_validate_batch(const ekv_pool* pool, const ekv_batch* batch, int32_t* report, hipStream_t stream) {
  ekv::ValidateBatchArgs a{batch->seq_lens, batch->block_table, batch->tags,
                           batch->mode == EKV_MODE_NATIVE ? nullptr : batch->boundaries, report,
                           batch->batch, batch->max_blocks, pool->num_blocks, batch->max_seq_len, batch->mode};
  return ekv::launch_validate_batch(a, stream);
}

// The report buffer of the debug mode: a static device array (one per
// device, looked up like the scratch above), so that the debug mode
// allocates nothing either.  Debug-mode calls synchronise before they read
// it; calls that overlap on one device from several host threads race on it.
static __device__ __align__(16) int32_t debug_report[2 * EKV_VIOL_COUNT];

ekv_status debug_report_buffer(int32_t** out) {
  static std::mutex mu;
  static void* addr[kScratchDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return hip_status(hipGetLastError(), "hipGetDevice");
  if (dev < 0 || dev >= kScratchDevices) return fail(EKV_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kScratchDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(debug_report));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(debug_report)");
    addr[dev] = ptr;
  }
  *out = static_cast<int32_t*>(addr[dev]);
  return EKV_OK;
}

// Waits for the checks enqueued on the stream and turns the first reported
// violation into EKV_ERR_INVALID.
ekv_status debug_verdict(const int32_t* report, hipStream_t stream, const char* call) {
  int32_t h[2 * EKV_VIOL_COUNT];
  hipError_t e = hipMemcpyAsync(h, report, sizeof h, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_status(e, "EKV_DEBUG report read");
  for (int k = 0; k < EKV_VIOL_COUNT; ++k)
    if (h[k] > 0)
      return fail(EKV_ERR_INVALID, "%s (EKV_DEBUG): %d violation(s): %s; first at index %d", call, h[k],
                  violation_name(k), h[EKV_VIOL_COUNT + k]);
  return EKV_OK;
}

ekv_status debug_check_batch(const ekv_pool* pool, const ekv_batch* batch, hipStream_t stream, const char* call) {
  if ((long long)batch->batch * batch->max_blocks >= (1LL << 31))
    return fail(EKV_ERR_UNSUPPORTED, "%s (EKV_DEBUG): batch * max_blocks must be below 2^31", call);
  int32_t* report = nullptr;
  ekv_status st = debug_report_buffer(&report);
  if (st != EKV_OK) return st;
  if ((st = hip_status(enqueue_validate_batch(pool, batch, report, stream), "EKV_DEBUG check launch")) != EKV_OK)
    return st;
  return debug_verdict(report, stream, call);
}

ekv_status debug_check_list(const ekv_pool* pool, int kind, int n, const int32_t* pairs, const int32_t* new_blocks,
                            const int32_t* block_table, const uint8_t* tags, int batch, int max_blocks,
                            hipStream_t stream, const char* call) {
  int32_t* report = nullptr;
  ekv_status st = debug_report_buffer(&report);
  if (st != EKV_OK) return st;
  ekv::ValidateListArgs a{pairs, new_blocks, block_table, tags, nullptr, report, n, kind, batch, max_blocks,
                          pool->num_blocks};
  if ((st = hip_status(ekv::launch_validate_list(a, stream), "EKV_DEBUG check launch")) != EKV_OK) return st;
  return debug_verdict(report, stream, call);
}

// One decode call on a workspace: the caller's, or (clear_counters) the
// static scratch, whose merge counters are zeroed first by a fill kernel;
// that call runs no EKV_DEBUG checks (they synchronise the stream, which
// its callers -- graph capture among them -- cannot have).
ekv_status decode_call(const ekv_pool* pool, const ekv_batch* batch, const void* q, void* out, int32_t out_dtype,
                       float scale, void* ws, size_t ws_bytes, bool clear_counters, hipStream_t stream,
                       const char* who, const void* k_new = nullptr, const void* v_new = nullptr) {
  ekv_status st = check_pool(pool);
  if (st != EKV_OK) return st;
  int group = 0;
  if ((st = check_attention_batch(pool, batch, &group)) != EKV_OK) return st;
  if (batch->batch == 0) return EKV_OK;
  if (!q || !out) return fail(EKV_ERR_INVALID, "q and out are required");
  if ((k_new == nullptr) != (v_new == nullptr)) return fail(EKV_ERR_INVALID, "%s: k_new and v_new go together", who);
  const int q_dtype = pool->dtype == EKV_DTYPE_E5M2 ? EKV_DTYPE_FP16 : pool->dtype;   // 8-bit pools: FP16 queries
  if (out_dtype != q_dtype && out_dtype != EKV_DTYPE_FP32)
    return fail(EKV_ERR_INVALID, "out_dtype must be the query dtype or fp32");
  if (!std::isfinite(scale)) return fail(EKV_ERR_INVALID, "scale must be finite");
  DecodePlan plan{};
  if (!clear_counters) {   // the caller's workspace: at least ekv_decode_workspace_bytes
    if ((st = plan_decode(pool, batch, group, false, &plan)) != EKV_OK) return st;
    if (!ws || ws_bytes < plan.total)
      return fail(EKV_ERR_INVALID, "workspace of %zu bytes needed, %zu given", plan.total, ws_bytes);
    if (reinterpret_cast<uintptr_t>(ws) % 16)   // the partial rows move in 16-byte accesses
      return fail(EKV_ERR_INVALID, "%s: ws must be 16-byte aligned", who);
  }
  if ((st = plan_decode(pool, batch, group, true, &plan)) != EKV_OK) return st;
  if (plan.total > ws_bytes)   // (the static scratch: sized by the device's own grid)
    return fail(EKV_ERR_UNSUPPORTED, "%s: needs %zu bytes of scratch, %zu available", who, plan.total, ws_bytes);
  // (the debug checks synchronise: not for the no-allocation call)
  if (!clear_counters && debug_mode() && (st = debug_check_batch(pool, batch, stream, who)) != EKV_OK) return st;
  const bool elastic = batch->mode != EKV_MODE_NATIVE;
  ekv::DecodeArgs a{};
  a.pool = static_cast<const uint16_t*>(pool->kv);
  a.q = static_cast<const uint16_t*>(q);
  a.seq_lens = batch->seq_lens;
  a.bt = batch->block_table;
  a.tags = batch->tags;
  a.bounds = elastic ? batch->boundaries : nullptr;
  a.counters = static_cast<uint32_t*>(ws);
  a.ws_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + plan.ml_offset);
  a.ws_o = reinterpret_cast<float*>(static_cast<char*>(ws) + plan.o_offset);
  a.out = out;
  a.batch = batch->batch;
  a.num_kv_heads = pool->num_kv_heads;
  a.num_q_heads = batch->num_q_heads;
  a.max_blocks = batch->max_blocks;
  a.num_blocks = pool->num_blocks;
  a.len_cap = max_seq_blocks(batch) * ekv::kPage;
  if (batch->max_seq_len > 0) a.len_cap = std::min(a.len_cap, batch->max_seq_len);
  a.min_chunk = plan.min_chunk;
  a.pairs_max = plan.pairs_max;
  a.grid = plan.grid;
  a.out_fp32 = out_dtype == EKV_DTYPE_FP32;
  a.slots = decode_slots(pool, group, elastic);
  a.scale_log2 = log2e_scale(scale);
  a.k_new = k_new;
  a.v_new = v_new;
  a.pool_out = k_new ? pool->kv : nullptr;
  if (clear_counters &&
      (st = hip_status(ekv::launch_zero_u32(a.counters, 2 * (size_t)plan.grid, stream), "scratch clear")) != EKV_OK)
    return st;
  return hip_status(ekv::launch_decode(a, pool->dtype, group, elastic, stream), "decode launch");
}

}  // namespace

extern "C" {

const char* ekv_status_string(ekv_status s) {
  switch (s) {
    case EKV_OK: return "ok";
    case EKV_ERR_INVALID: return "invalid argument";
    case EKV_ERR_UNSUPPORTED: return "unsupported";
    case EKV_ERR_HIP: return "HIP runtime error";
    case EKV_ERR_HOST: return "host-side failure";
    default: return "unknown status";
  }
}

const char* ekv_last_error(void) { return g_last_error; }

const char* ekv_version(void) { return "0.1.0"; }

ekv_status ekv_lower(const uint8_t* h_tags, const int32_t* h_seq_lens, int32_t batch,
                     int32_t max_blocks, int32_t page_size, int32_t* mode_out,
                     int32_t* h_boundaries_out) {
  return ekv::guard("ekv_lower", [&]() -> ekv_status {
    if (!mode_out || batch < 0 || max_blocks <= 0 || page_size <= 0)
      return fail(EKV_ERR_INVALID, "ekv_lower: bad sizes or NULL mode_out");
    if (batch > 0 && (!h_tags || !h_seq_lens || !h_boundaries_out))
      return fail(EKV_ERR_INVALID, "ekv_lower: NULL array");
    bool any_base = false, any_irregular = false;
    for (int s = 0; s < batch; ++s) {
      const int len = h_seq_lens[s];
      if (len < 0 || (long long)len > (long long)max_blocks * page_size)
        return fail(EKV_ERR_INVALID, "ekv_lower: sequence %d length %d out of range", s, len);
      const int nblk = (len + page_size - 1) / page_size;
      const uint8_t* row = h_tags + (size_t)s * max_blocks;
      int first = -1, last = -1, count = 0;
      int j = 0;
      // four full pairs (8 tag bytes) per step: every byte 0 or 1, the two
      // bytes of each pair equal, and member 0's low bit marks a BASE pair;
      // a word that fails a test is redone byte by byte below for the message
      for (; 2 * j + 8 <= nblk; j += 4) {
        uint64_t w;
        std::memcpy(&w, row + 2 * j, 8);
        if ((w & 0xFEFEFEFEFEFEFEFEull) || ((w ^ (w >> 8)) & 0x00FF00FF00FF00FFull)) break;
        const uint64_t m = w & 0x0001000100010001ull;   // bit 16k: pair j + k is BASE
        // selects, not branches: the BASE pattern is data and mispredicts
        const int lo = j + __builtin_ctzll(m | (1ull << 63)) / 16;
        const int hi = j + (63 - __builtin_clzll(m | 1ull)) / 16;
        first = (first < 0 && m) ? lo : first;
        last = m ? hi : last;
        count += __builtin_popcountll(m);
      }
      for (; 2 * j < nblk; ++j) {
        const uint8_t a = row[2 * j];
        const uint8_t b = (2 * j + 1 < nblk) ? row[2 * j + 1] : a;
        if (a > 1 || b > 1) return fail(EKV_ERR_INVALID, "ekv_lower: tag value out of range");
        if (a != b) return fail(EKV_ERR_INVALID, "ekv_lower: pair %d of sequence %d has mixed tags", j, s);
        if (a) {
          if (first < 0) first = j;
          last = j;
          ++count;
        }
      }
      int32_t* out = h_boundaries_out + 2 * s;
      if (count == 0) {
        out[0] = out[1] = 0;
      } else if (count == last - first + 1) {
        any_base = true;
        out[0] = first;
        out[1] = last + 1;
      } else {
        any_base = any_irregular = true;
        out[0] = out[1] = -1;
      }
    }
    *mode_out = !any_base ? EKV_MODE_NATIVE : (any_irregular ? EKV_MODE_GENERAL : EKV_MODE_STRUCTURED);
    return EKV_OK;
  });
}

size_t ekv_decode_workspace_bytes(const ekv_pool* pool, const ekv_batch* batch) {
  int group = 0;   // (no allocation or exception on this path)
  if (check_pool(pool) != EKV_OK || check_attention_batch(pool, batch, &group) != EKV_OK) return 0;
  DecodePlan plan{};
  if (plan_decode(pool, batch, group, false, &plan) != EKV_OK) return 0;
  return plan.total;
}

ekv_status ekv_decode_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream) {
  return ekv::guard("ekv_decode_workspace_init", [&]() -> ekv_status {
    if (!ws && ws_bytes) return fail(EKV_ERR_INVALID, "ws is NULL");
    if (ws_bytes % 4) return fail(EKV_ERR_INVALID, "ws_bytes must be a multiple of 4");
    return hip_status(ekv::launch_zero_u32(static_cast<uint32_t*>(ws), ws_bytes / 4, stream),
                      "ekv_decode_workspace_init launch");
  });
}

ekv_status ekv_attn_decode(const ekv_pool* pool, const ekv_batch* batch, const void* q, void* out,
                           int32_t out_dtype, float scale, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  return ekv::guard("ekv_attn_decode", [&]() -> ekv_status {
    return decode_call(pool, batch, q, out, out_dtype, scale, ws, ws_bytes, false, stream, "ekv_attn_decode");
  });
}

ekv_status ekv_attn_decode_append(const ekv_pool* pool, const ekv_batch* batch, const void* q, const void* k_new,
                                  const void* v_new, void* out, int32_t out_dtype, float scale, void* ws,
                                  size_t ws_bytes, hipStream_t stream) {
  return ekv::guard("ekv_attn_decode_append", [&]() -> ekv_status {
    if (!k_new || !v_new) return fail(EKV_ERR_INVALID, "ekv_attn_decode_append: k_new and v_new are required");
    return decode_call(pool, batch, q, out, out_dtype, scale, ws, ws_bytes, false, stream, "ekv_attn_decode_append",
                       k_new, v_new);
  });
}

ekv_status ekv_attn_decode_noalloc(const ekv_pool* pool, const ekv_batch* batch, const void* q, void* out,
                                   int32_t out_dtype, float scale, hipStream_t stream) {
  return ekv::guard("ekv_attn_decode_noalloc", [&]() -> ekv_status {
    void* ws = nullptr;
    const ekv_status st = scratch_address(&ws);
    if (st != EKV_OK) return st;
    return decode_call(pool, batch, q, out, out_dtype, scale, ws, kScratchBytes, true, stream,
                       "ekv_attn_decode_noalloc");
  });
}

ekv_status ekv_attn_prefill(const ekv_pool* pool, const ekv_batch* batch, const void* q,
                            const int32_t* cu_q, int32_t total_q, int32_t max_q_len, void* out,
                            int32_t out_dtype, float scale, hipStream_t stream) {
  return ekv::guard("ekv_attn_prefill", [&]() -> ekv_status {
    ekv_status st = check_pool(pool);
    if (st != EKV_OK) return st;
    int group = 0;
    if ((st = check_attention_batch(pool, batch, &group)) != EKV_OK) return st;
    if (total_q < 0 || max_q_len < 0) return fail(EKV_ERR_INVALID, "negative sizes");
    if (batch->batch == 0 || total_q == 0) return EKV_OK;
    if (!q || !out || !cu_q) return fail(EKV_ERR_INVALID, "q, cu_q and out are required");
    const int q_dtype = pool->dtype == EKV_DTYPE_E5M2 ? EKV_DTYPE_FP16 : pool->dtype;   // 8-bit pools: FP16 queries
    if (out_dtype != q_dtype && out_dtype != EKV_DTYPE_FP32)
      return fail(EKV_ERR_INVALID, "out_dtype must be the query dtype or fp32");
    if (!std::isfinite(scale)) return fail(EKV_ERR_INVALID, "scale must be finite");
    if (max_q_len == 0) return EKV_OK;
    if (debug_mode() && (st = debug_check_batch(pool, batch, stream, "ekv_attn_prefill")) != EKV_OK) return st;
    ekv::PrefillArgs a{};
    a.pool = static_cast<const uint16_t*>(pool->kv);
    a.q = static_cast<const uint16_t*>(q);
    a.cu_q = cu_q;
    a.seq_lens = batch->seq_lens;
    a.bt = batch->block_table;
    a.tags = batch->tags;
    a.bounds = batch->mode == EKV_MODE_NATIVE ? nullptr : batch->boundaries;
    a.out = out;
    a.batch = batch->batch;
    a.num_kv_heads = pool->num_kv_heads;
    a.num_q_heads = batch->num_q_heads;
    a.max_blocks = batch->max_blocks;
    a.max_q_len = max_q_len;
    a.num_blocks = pool->num_blocks;
    a.total_q = total_q;
    a.out_fp32 = out_dtype == EKV_DTYPE_FP32;
    a.scale_log2 = log2e_scale(scale);
    return hip_status(ekv::launch_prefill(a, pool->dtype, group, batch->mode != EKV_MODE_NATIVE, stream),
                      "ekv_attn_prefill launch");
  });
}

ekv_status ekv_append_kv(const ekv_pool* pool, const int32_t* slots, const void* k, const void* v,
                         int32_t n, hipStream_t stream) {
  return ekv::guard("ekv_append_kv", [&]() -> ekv_status {
    ekv_status st = check_pool(pool);
    if (st != EKV_OK) return st;
    if (n < 0) return fail(EKV_ERR_INVALID, "negative n");
    if (n == 0) return EKV_OK;
    if (!slots || !k || !v) return fail(EKV_ERR_INVALID, "slots, k and v are required");
    ekv::AppendArgs a{static_cast<uint16_t*>(pool->kv), slots, static_cast<const uint16_t*>(k),
                      static_cast<const uint16_t*>(v), n, pool->num_kv_heads, pool->dtype == EKV_DTYPE_E5M2,
                      pool->num_blocks};
    return hip_status(ekv::launch_append(a, stream), "ekv_append_kv launch");
  });
}

static ekv_status check_transition_args(const ekv_pool* pool, int32_t n, const int32_t* pairs,
                                        int32_t* block_table, uint8_t* tags, int32_t batch,
                                        int32_t max_blocks) {
  ekv_status st = check_pool(pool);
  if (st != EKV_OK) return st;
  if (n < 0 || batch < 0 || max_blocks < 2) return fail(EKV_ERR_INVALID, "bad sizes");
  if (n > 0 && (!pairs || !block_table || !tags))
    return fail(EKV_ERR_INVALID, "pairs, block_table and tags are required");
  if (n > 65535) return fail(EKV_ERR_UNSUPPORTED, "at most 65535 pairs per call");
  return EKV_OK;
}

// The device address of [p, p + bytes) if the whole range is memory the
// current device can read (its own memory, or pinned host memory mapped for
// it), else an error.  Both ends are looked up: they must lie in memory the
// runtime knows and map to device addresses exactly bytes - 1 apart.
static ekv_status device_readable(const void* p, size_t bytes, int device, const uint8_t** out) {
  hipPointerAttribute_t a0{}, a1{};
  const char* last = static_cast<const char*>(p) + bytes - 1;
  const bool known = hipPointerGetAttributes(&a0, p) == hipSuccess && hipPointerGetAttributes(&a1, last) == hipSuccess;
  if (!known) {
    (void)hipGetLastError();   // the failed lookup must not surface as a launch error
    return fail(EKV_ERR_INVALID, "source %p is not memory the device can read (unpinned host memory?)", p);
  }
  for (const hipPointerAttribute_t* a : {&a0, &a1}) {
    const bool ok = (a->type == hipMemoryTypeHost || (a->type == hipMemoryTypeDevice && a->device == device)) &&
                    a->devicePointer != nullptr;
    if (!ok) return fail(EKV_ERR_INVALID, "source %p is not mapped for the current device", p);
  }
  const char* d0 = static_cast<const char*>(a0.devicePointer);
  const char* d1 = static_cast<const char*>(a1.devicePointer);
  if (d1 - d0 != static_cast<ptrdiff_t>(bytes - 1))
    return fail(EKV_ERR_INVALID, "source %p does not cover one block's bytes in one mapping", p);
  *out = reinterpret_cast<const uint8_t*>(d0);
  return EKV_OK;
}

// Refinement bytes live in device memory of the current device or in pinned
// host memory mapped for it (the CPU backing); the range is checked at both
// ends with device_readable and replaced by its device address.  Anything
// else -- pageable host memory, another device's memory, memory the runtime
// cannot describe -- is EKV_ERR_INVALID before anything is enqueued, so the
// kernels never touch memory they cannot reach.
static ekv_status resolve_lo(const uint8_t* p, size_t bytes, const uint8_t** out) {
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) return hip_status(hipGetLastError(), "hipGetDevice");
  return device_readable(p, bytes, device, out);
}

static size_t block_bytes_of(const ekv_pool* pool) {
  return (size_t)2 * pool->num_kv_heads * pool->page_size * pool->head_dim * (pool->dtype == EKV_DTYPE_E5M2 ? 1 : 2);
}

ekv_status ekv_demote(const ekv_pool* pool, int32_t n, const int32_t* pairs, int32_t* block_table,
                      uint8_t* tags, int32_t batch, int32_t max_blocks, int32_t* freed_out,
                      uint8_t* lo_out, hipStream_t stream) {
  return ekv::guard("ekv_demote", [&]() -> ekv_status {
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (n == 0) return EKV_OK;
    if (!freed_out) return fail(EKV_ERR_INVALID, "freed_out is required");
    const uint8_t* lo = nullptr;
    if (lo_out && (st = resolve_lo(lo_out, (size_t)n * block_bytes_of(pool), &lo)) != EKV_OK) return st;
    if (debug_mode() &&
        (st = debug_check_list(pool, 0, n, pairs, nullptr, block_table, tags, batch, max_blocks, stream, "ekv_demote")) != EKV_OK)
      return st;
    ekv::TransitionArgs a{static_cast<uint16_t*>(pool->kv), nullptr, pairs, nullptr, block_table, tags,
                          freed_out, const_cast<uint8_t*>(lo), n, pool->num_kv_heads, max_blocks, 1, 0, pool->dtype == EKV_DTYPE_E5M2, batch, pool->num_blocks};
    return hip_status(ekv::launch_demote(a, stream), "ekv_demote launch");
  });
}

ekv_status ekv_demote_layers(const ekv_pool* pool, const uint64_t* layer_kv, int32_t num_layers, int32_t n,
                             const int32_t* pairs, int32_t* block_table, uint8_t* tags, int32_t batch,
                             int32_t max_blocks, int32_t* freed_out, uint8_t* lo_out, hipStream_t stream) {
  return ekv::guard("ekv_demote_layers", [&]() -> ekv_status {
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (!layer_kv || num_layers < 1 || num_layers > 65535)
      return fail(EKV_ERR_INVALID, "layer_kv is required and num_layers must be in [1, 65535]");
    if (n == 0) return EKV_OK;
    if (!freed_out) return fail(EKV_ERR_INVALID, "freed_out is required");
    const uint8_t* lo = nullptr;
    if (lo_out && (st = resolve_lo(lo_out, (size_t)n * num_layers * block_bytes_of(pool), &lo)) != EKV_OK) return st;
    if (debug_mode() && (st = debug_check_list(pool, 0, n, pairs, nullptr, block_table, tags, batch, max_blocks, stream,
                                               "ekv_demote_layers")) != EKV_OK)
      return st;
    ekv::TransitionArgs a{nullptr, layer_kv, pairs, nullptr, block_table, tags,
                          freed_out, const_cast<uint8_t*>(lo), n, pool->num_kv_heads, max_blocks, num_layers, 0, pool->dtype == EKV_DTYPE_E5M2, batch, pool->num_blocks};
    return hip_status(ekv::launch_demote(a, stream), "ekv_demote_layers launch");
  });
}

ekv_status ekv_refine(const ekv_pool* pool, int32_t n, const int32_t* pairs,
                      const int32_t* new_blocks, int32_t* block_table, uint8_t* tags, int32_t batch,
                      int32_t max_blocks, const uint8_t* lo_in, hipStream_t stream) {
  return ekv::guard("ekv_refine", [&]() -> ekv_status {
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (n == 0) return EKV_OK;
    if (!new_blocks || !lo_in) return fail(EKV_ERR_INVALID, "new_blocks and lo_in are required");
    const uint8_t* lo = nullptr;
    st = resolve_lo(lo_in, (size_t)n * block_bytes_of(pool), &lo);
    if (st != EKV_OK) return st;
    if (debug_mode() &&
        (st = debug_check_list(pool, 1, n, pairs, new_blocks, block_table, tags, batch, max_blocks, stream, "ekv_refine")) != EKV_OK)
      return st;
    ekv::TransitionArgs a{static_cast<uint16_t*>(pool->kv), nullptr, pairs, new_blocks, block_table, tags,
                          nullptr, const_cast<uint8_t*>(lo), n, pool->num_kv_heads, max_blocks, 1, 0, pool->dtype == EKV_DTYPE_E5M2, batch, pool->num_blocks};
    return hip_status(ekv::launch_refine(a, stream), "ekv_refine launch");
  });
}

ekv_status ekv_refine_staged(const ekv_pool* pool, int32_t n, const int32_t* pairs, const int32_t* new_blocks,
                             int32_t* block_table, uint8_t* tags, int32_t batch, int32_t max_blocks,
                             hipStream_t stream) {
  return ekv::guard("ekv_refine_staged", [&]() -> ekv_status {
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (n == 0) return EKV_OK;
    if (!new_blocks) return fail(EKV_ERR_INVALID, "new_blocks is required");
    if (debug_mode() && (st = debug_check_list(pool, 1, n, pairs, new_blocks, block_table, tags, batch, max_blocks, stream,
                                               "ekv_refine_staged")) != EKV_OK)
      return st;
    ekv::TransitionArgs a{static_cast<uint16_t*>(pool->kv), nullptr, pairs, new_blocks, block_table, tags,
                          nullptr, nullptr, n, pool->num_kv_heads, max_blocks, 1, 1, pool->dtype == EKV_DTYPE_E5M2, batch, pool->num_blocks};
    return hip_status(ekv::launch_refine(a, stream), "ekv_refine_staged launch");
  });
}

ekv_status ekv_stage_blocks(const ekv_pool* pool, int32_t n, const void* const* h_src,
                            const int32_t* h_new_blocks, hipStream_t stream) {
  return ekv::guard("ekv_stage_blocks", [&]() -> ekv_status {
    ekv_status st = check_pool(pool);
    if (st != EKV_OK) return st;
    if (n < 0) return fail(EKV_ERR_INVALID, "negative n");
    if (n == 0) return EKV_OK;
    if (!h_src || !h_new_blocks) return fail(EKV_ERR_INVALID, "h_src and h_new_blocks are required");
    const int64_t block_bytes = (int64_t)block_bytes_of(pool);
    std::vector<uint8_t> used((size_t)pool->num_blocks, 0);
    for (int i = 0; i < n; ++i) {
      const int b = h_new_blocks[i];
      if (b < 0 || b >= pool->num_blocks) return fail(EKV_ERR_INVALID, "new block %d out of range", b);
      if (used[b]) return fail(EKV_ERR_INVALID, "new block %d listed twice", b);
      used[b] = 1;
      if (!h_src[i]) return fail(EKV_ERR_INVALID, "source %d is NULL", i);
    }
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess) return hip_status(hipGetLastError(), "hipGetDevice");
    // every source is checked before anything is enqueued
    std::vector<const uint8_t*> dev((size_t)n);
    for (int i = 0; i < n; ++i) {
      st = device_readable(h_src[i], (size_t)block_bytes, device, &dev[i]);
      if (st != EKV_OK) return st;
    }
    for (int first = 0; first < n; first += ekv::kStageMax) {
      ekv::StageArgs a{};
      a.pool = static_cast<uint8_t*>(pool->kv);
      a.block_bytes = block_bytes;
      a.n = std::min(n - first, ekv::kStageMax);
      for (int k = 0; k < a.n; ++k) {
        a.src[k] = dev[first + k];
        a.dst[k] = h_new_blocks[first + k];
      }
      st = hip_status(ekv::launch_stage(a, stream), "ekv_stage_blocks launch");
      if (st != EKV_OK) return st;
    }
    return EKV_OK;
  });
}

ekv_status ekv_promote_begin(const ekv_pool* pool, int32_t n, const void* const* h_src,
                             const int32_t* h_new_blocks, hipEvent_t copied, hipStream_t copy_stream) {
  return ekv::guard("ekv_promote_begin", [&]() -> ekv_status {
    if (!copied) return fail(EKV_ERR_INVALID, "ekv_promote_begin: the completion event is required");
    const ekv_status st = ekv_stage_blocks(pool, n, h_src, h_new_blocks, copy_stream);
    if (st != EKV_OK) return st;
    return hip_status(hipEventRecord(copied, copy_stream), "ekv_promote_begin event record");
  });
}

ekv_status ekv_promote_publish(const ekv_pool* pool, int32_t n, const int32_t* pairs, const int32_t* new_blocks,
                               int32_t* block_table, uint8_t* tags, int32_t batch, int32_t max_blocks,
                               hipEvent_t copied, hipStream_t stream) {
  return ekv::guard("ekv_promote_publish", [&]() -> ekv_status {
    if (!copied) return fail(EKV_ERR_INVALID, "ekv_promote_publish: the completion event is required");
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (n > 0 && !new_blocks) return fail(EKV_ERR_INVALID, "new_blocks is required");
    if ((st = hip_status(hipStreamWaitEvent(stream, copied, 0), "ekv_promote_publish wait")) != EKV_OK) return st;
    return ekv_refine_staged(pool, n, pairs, new_blocks, block_table, tags, batch, max_blocks, stream);
  });
}

ekv_status ekv_refine_layers(const ekv_pool* pool, const uint64_t* layer_kv, int32_t num_layers, int32_t n,
                             const int32_t* pairs, const int32_t* new_blocks, int32_t* block_table,
                             uint8_t* tags, int32_t batch, int32_t max_blocks, const uint8_t* lo_in,
                             hipStream_t stream) {
  return ekv::guard("ekv_refine_layers", [&]() -> ekv_status {
    ekv_status st = check_transition_args(pool, n, pairs, block_table, tags, batch, max_blocks);
    if (st != EKV_OK) return st;
    if (!layer_kv || num_layers < 1 || num_layers > 65535)
      return fail(EKV_ERR_INVALID, "layer_kv is required and num_layers must be in [1, 65535]");
    if (n == 0) return EKV_OK;
    if (!new_blocks || !lo_in) return fail(EKV_ERR_INVALID, "new_blocks and lo_in are required");
    const uint8_t* lo = nullptr;
    st = resolve_lo(lo_in, (size_t)n * num_layers * block_bytes_of(pool), &lo);
    if (st != EKV_OK) return st;
    if (debug_mode() && (st = debug_check_list(pool, 1, n, pairs, new_blocks, block_table, tags, batch, max_blocks, stream,
                                               "ekv_refine_layers")) != EKV_OK)
      return st;
    ekv::TransitionArgs a{nullptr, layer_kv, pairs, new_blocks, block_table, tags,
                          nullptr, const_cast<uint8_t*>(lo), n, pool->num_kv_heads, max_blocks, num_layers, 0, pool->dtype == EKV_DTYPE_E5M2, batch, pool->num_blocks};
    return hip_status(ekv::launch_refine(a, stream), "ekv_refine_layers launch");
  });
}

ekv_status ekv_check_transition(int32_t kind, const int32_t* h_pairs, int32_t n,
                                const int32_t* h_block_table, const uint8_t* h_tags,
                                const int32_t* h_seq_lens, int32_t batch, int32_t max_blocks,
                                int32_t page_size, int32_t num_blocks,
                                const int32_t* h_new_blocks) {
  return ekv::guard("ekv_check_transition", [&]() -> ekv_status {
    if (kind != 0 && kind != 1) return fail(EKV_ERR_INVALID, "kind must be 0 (demote) or 1 (refine)");
    if (n < 0 || batch < 0 || max_blocks < 2 || page_size <= 0 || num_blocks <= 0)
      return fail(EKV_ERR_INVALID, "bad sizes");
    if (n == 0) return EKV_OK;
    if (!h_pairs || !h_block_table || !h_tags || !h_seq_lens)
      return fail(EKV_ERR_INVALID, "NULL host mirror");
    const uint8_t want = kind == 0 ? EKV_TAG_TARGET : EKV_TAG_BASE;
    std::vector<uint8_t> seen((size_t)batch * max_blocks, 0);
    for (int i = 0; i < n; ++i) {
      const int s = h_pairs[2 * i], j = h_pairs[2 * i + 1];
      if (s < 0 || s >= batch || j < 0 || 2 * j + 1 >= max_blocks)
        return fail(EKV_ERR_INVALID, "pair %d (%d,%d) out of range", i, s, j);
      if ((long long)2 * page_size * (j + 1) > h_seq_lens[s])
        return fail(EKV_ERR_INVALID, "pair %d (%d,%d) is not two full blocks", i, s, j);
      uint8_t& mark = seen[(size_t)s * max_blocks + 2 * j];
      if (mark) return fail(EKV_ERR_INVALID, "pair (%d,%d) listed twice", s, j);
      mark = 1;
      const uint8_t* row = h_tags + (size_t)s * max_blocks;
      if (row[2 * j] != want || row[2 * j + 1] != want)
        return fail(EKV_ERR_INVALID, "pair (%d,%d) is not in the expected state", s, j);
      const int32_t* bt = h_block_table + (size_t)s * max_blocks;
      for (int m = 0; m < 2; ++m)
        if (bt[2 * j + m] < 0 || bt[2 * j + m] >= num_blocks)
          return fail(EKV_ERR_INVALID, "pair (%d,%d) maps outside the pool", s, j);
    }
    if (kind == 1) {
      if (!h_new_blocks) return fail(EKV_ERR_INVALID, "refinement needs new blocks");
      std::vector<uint8_t> used((size_t)num_blocks, 0);
      for (int s = 0; s < batch; ++s) {
        const int nblk = (h_seq_lens[s] + page_size - 1) / page_size;
        for (int i = 0; i < nblk && i < max_blocks; ++i) {
          const int b = h_block_table[(size_t)s * max_blocks + i];
          if (b >= 0 && b < num_blocks) used[b] = 1;
        }
      }
      for (int i = 0; i < n; ++i) {
        const int b = h_new_blocks[i];
        if (b < 0 || b >= num_blocks) return fail(EKV_ERR_INVALID, "new block %d out of range", b);
        if (used[b]) return fail(EKV_ERR_INVALID, "new block %d is in use", b);
        used[b] = 1;
      }
    }
    return EKV_OK;
  });
}

ekv_status ekv_validate_batch(const ekv_pool* pool, const ekv_batch* batch, int32_t* report, hipStream_t stream) {
  return ekv::guard("ekv_validate_batch", [&]() -> ekv_status {
    const ekv_status st = check_validate_batch(pool, batch, report);
    if (st != EKV_OK) return st;
    return hip_status(enqueue_validate_batch(pool, batch, report, stream), "ekv_validate_batch launch");
  });
}

ekv_status ekv_validate_transition(const ekv_pool* pool, int32_t kind, int32_t n, const int32_t* pairs,
                                   const int32_t* new_blocks, const int32_t* block_table, const uint8_t* tags,
                                   const int32_t* seq_lens, int32_t batch, int32_t max_blocks, int32_t* report,
                                   hipStream_t stream) {
  return ekv::guard("ekv_validate_transition", [&]() -> ekv_status {
    const ekv_status st = check_pool(pool);
    if (st != EKV_OK) return st;
    if (kind != 0 && kind != 1) return fail(EKV_ERR_INVALID, "kind must be 0 (demotion) or 1 (refinement)");
    if (n < 0 || batch < 0 || max_blocks < 2) return fail(EKV_ERR_INVALID, "bad sizes");
    if (!report) return fail(EKV_ERR_INVALID, "report is required");
    if (n > 0 && (!pairs || !block_table || !tags)) return fail(EKV_ERR_INVALID, "pairs, block_table and tags are required");
    if ((long long)batch * max_blocks >= (1LL << 31))
      return fail(EKV_ERR_UNSUPPORTED, "batch * max_blocks must be below 2^31");
    ekv::ValidateListArgs a{pairs, kind == 1 ? new_blocks : nullptr, block_table, tags, seq_lens, report, n, kind,
                            batch, max_blocks, pool->num_blocks};
    return hip_status(ekv::launch_validate_list(a, stream), "ekv_validate_transition launch");
  });
}

}  // extern "C"
