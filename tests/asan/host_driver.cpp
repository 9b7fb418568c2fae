// Host-side exercise of libekv's C++ under AddressSanitizer (and the
// undefined-behaviour checker): the metadata lowering and its word scans,
// the transition-list checks, the controller, the argument checks of every
// device entry point (which return before any device work here) and the
// pointer lookups of the refinement-byte and staging paths (which find no
// device on a CPU-only machine).  Every array is a heap allocation of the
// exact size the interface documents, so a read or write past it is
// reported.  Prints "host driver ok" and returns 0 when every call behaved.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "ekv.h"

namespace {

int failures = 0;

void expect(bool ok, const char* what, int k) {
  if (!ok) {
    std::fprintf(stderr, "FAILED: %s (case %d): %s\n", what, k, ekv_last_error());
    ++failures;
  }
}

template <typename T>
T* exact(size_t n) {   // an allocation of exactly n elements (never zero bytes)
  return static_cast<T*>(std::malloc(n ? n * sizeof(T) : 1));
}

// Lowering: random tag tables, rows whose block count is exactly the table
// width (so the 8-byte word scan of the last row ends at the allocation's end).
void lowering(std::mt19937& rng) {
  for (int k = 0; k < 3000; ++k) {
    const int batch = 1 + rng() % 9, max_blocks = 1 + rng() % 70;
    uint8_t* tags = exact<uint8_t>((size_t)batch * max_blocks);
    int32_t* lens = exact<int32_t>(batch);
    int32_t* bounds = exact<int32_t>(2 * (size_t)batch);
    for (int s = 0; s < batch; ++s) {
      lens[s] = (rng() % 4 == 0) ? max_blocks * 16 : (int32_t)(rng() % (max_blocks * 16 + 1));
      const int nblk = (lens[s] + 15) / 16;
      for (int j = 0; j < max_blocks; j += 2) {
        const uint8_t t = (rng() % 3 == 0) ? 1 : 0;
        tags[s * max_blocks + j] = t;
        if (j + 1 < max_blocks) tags[s * max_blocks + j + 1] = (rng() % 50 == 0) ? (uint8_t)(1 - t) : t;
      }
      if (2 * (nblk / 2) < nblk) tags[s * max_blocks + nblk - 1] = 0;   // a lone last block is TARGET
      if (rng() % 40 == 0 && nblk) tags[s * max_blocks + rng() % nblk] = 2;   // bad value
    }
    int32_t mode = -1;
    const ekv_status st = ekv_lower(tags, lens, batch, max_blocks, 16, &mode, bounds);
    expect(st == EKV_OK || st == EKV_ERR_INVALID, "ekv_lower status", k);
    if (st == EKV_OK) expect(mode >= EKV_MODE_NATIVE && mode <= EKV_MODE_GENERAL, "ekv_lower mode", k);
    std::free(tags);
    std::free(lens);
    std::free(bounds);
  }
  int32_t mode = 0;
  expect(ekv_lower(nullptr, nullptr, 2, 4, 16, &mode, nullptr) == EKV_ERR_INVALID, "ekv_lower NULL", 0);
  expect(ekv_lower(nullptr, nullptr, 0, 4, 16, &mode, nullptr) == EKV_OK, "ekv_lower empty", 0);
}

// Transition-list checks on random mirrors and lists (valid and not).
void transitions(std::mt19937& rng) {
  for (int k = 0; k < 2000; ++k) {
    const int batch = 1 + rng() % 6, max_blocks = 2 + rng() % 40, num_blocks = batch * max_blocks + 8;
    int32_t* bt = exact<int32_t>((size_t)batch * max_blocks);
    uint8_t* tags = exact<uint8_t>((size_t)batch * max_blocks);
    int32_t* lens = exact<int32_t>(batch);
    for (int i = 0; i < batch * max_blocks; ++i) {
      bt[i] = (int32_t)(rng() % (num_blocks + 2)) - 1;
      tags[i] = (uint8_t)(rng() % 2);
    }
    for (int s = 0; s < batch; ++s) lens[s] = (int32_t)(rng() % (max_blocks * 16 + 1));
    const int n = rng() % 12;
    int32_t* pairs = exact<int32_t>(2 * (size_t)n);
    int32_t* fresh = exact<int32_t>(n);
    for (int i = 0; i < n; ++i) {
      pairs[2 * i] = (int32_t)(rng() % (batch + 1)) - (rng() % 9 == 0);
      pairs[2 * i + 1] = (int32_t)(rng() % (max_blocks / 2 + 1));
      fresh[i] = (int32_t)(rng() % (num_blocks + 2)) - 1;
    }
    for (int kind = 0; kind < 2; ++kind) {
      const ekv_status st = ekv_check_transition(kind, pairs, n, bt, tags, lens, batch, max_blocks, 16, num_blocks,
                                                 kind ? fresh : nullptr);
      expect(st == EKV_OK || st == EKV_ERR_INVALID, "ekv_check_transition status", k);
    }
    std::free(bt);
    std::free(tags);
    std::free(lens);
    std::free(pairs);
    std::free(fresh);
  }
}

// Controller: random demand sequences over random mirrors.
void controller(std::mt19937& rng) {
  for (int k = 0; k < 1000; ++k) {
    const int batch = 1 + rng() % 8, max_blocks = 2 + rng() % 64;
    uint8_t* tags = exact<uint8_t>((size_t)batch * max_blocks);
    uint8_t* backed = exact<uint8_t>((size_t)batch * max_blocks);
    int32_t* lens = exact<int32_t>(batch);
    for (int s = 0; s < batch; ++s) {
      lens[s] = (int32_t)(rng() % (max_blocks * 16 + 1));
      for (int j = 0; j < max_blocks; j += 2) {
        const uint8_t t = (uint8_t)(rng() % 2);
        tags[s * max_blocks + j] = t;
        if (j + 1 < max_blocks) tags[s * max_blocks + j + 1] = t;
      }
    }
    for (int i = 0; i < batch * max_blocks; ++i) backed[i] = (uint8_t)(rng() % 4 != 0);
    ekv_ctrl_config cfg{};
    cfg.min_batch = rng() % 20;
    cfg.decay = rng() % 4;
    cfg.a_max = (int32_t)(rng() % 200) - 20;
    cfg.sink_pairs = rng() % 3;
    cfg.recent_pairs = rng() % 3;
    cfg.policy = rng() % 2;
    cfg.watermark = rng() % 50;
    cfg.flags = rng() % 3;
    ekv_ctrl_state st{};
    const int max_pairs = rng() % 40;
    int32_t* out = exact<int32_t>(2 * (size_t)max_pairs);
    for (int step = 0; step < 5; ++step) {
      int32_t n = -1;
      ekv_status e = ekv_ctrl_demotion(&cfg, &st, rng() % 100, rng() % 100, tags, lens, (rng() % 2) ? backed : nullptr,
                                       batch, max_blocks, 16, out, max_pairs, &n);
      expect(e == EKV_OK || e == EKV_ERR_INVALID, "ekv_ctrl_demotion status", k);
      if (e == EKV_OK) expect(n >= 0 && n <= max_pairs, "demotion count", k);
      e = ekv_ctrl_promotion(&cfg, &st, rng() % 100, rng() % 50, tags, lens, batch, max_blocks, 16, out, max_pairs, &n);
      expect(e == EKV_OK || e == EKV_ERR_INVALID, "ekv_ctrl_promotion status", k);
      if (e == EKV_OK) expect(n >= 0 && n <= max_pairs, "promotion count", k);
    }
    std::free(tags);
    std::free(backed);
    std::free(lens);
    std::free(out);
  }
}

// Argument checks of the device entry points: every call here must return
// an error before any device work (no device exists on this machine, and
// the pointers are not device memory).
void arguments() {
  uint8_t* host = exact<uint8_t>(1 << 16);
  ekv_pool pool{host, 64, 2, 16, 128, EKV_DTYPE_BF16};
  int32_t* lens = exact<int32_t>(2);
  int32_t* bt = exact<int32_t>(8);
  ekv_batch batch{2, 8, 4, EKV_MODE_NATIVE, 0, lens, bt, nullptr, nullptr};
  const size_t need = ekv_decode_workspace_bytes(&pool, &batch);
  expect(need > 0, "workspace size", 0);
  expect(ekv_attn_decode(&pool, &batch, host, host, EKV_DTYPE_BF16, 1.f, host, need - 1, nullptr) == EKV_ERR_INVALID,
         "decode small workspace", 0);
  expect(ekv_attn_decode(&pool, &batch, host, host, EKV_DTYPE_BF16, 1.f, host + 8, need, nullptr) == EKV_ERR_INVALID,
         "decode misaligned workspace", 0);
  expect(ekv_attn_decode(nullptr, &batch, host, host, 0, 1.f, host, need, nullptr) == EKV_ERR_INVALID, "decode NULL", 0);
  expect(ekv_attn_decode(&pool, &batch, host, host, 0, NAN, host, need, nullptr) == EKV_ERR_INVALID, "decode scale", 0);
  expect(ekv_attn_decode_append(&pool, &batch, host, nullptr, host, host, 0, 1.f, host, need, nullptr) == EKV_ERR_INVALID,
         "decode_append without k_new", 0);
  expect(ekv_attn_decode_append(&pool, &batch, host, host, host, host, 0, 1.f, host, need - 1, nullptr) ==
             EKV_ERR_INVALID,
         "decode_append small workspace", 0);
  ekv_pool bad = pool;
  bad.head_dim = 64;
  expect(ekv_attn_prefill(&bad, &batch, host, lens, 1, 1, host, 0, 1.f, nullptr) == EKV_ERR_UNSUPPORTED, "prefill dim", 0);
  int32_t* pairs = exact<int32_t>(2);
  pairs[0] = 0;
  pairs[1] = 0;
  // refinement bytes in pageable host memory: rejected by the pointer checks
  const ekv_status d = ekv_demote(&pool, 1, pairs, bt, host, 2, 4, lens, host, nullptr);
  expect(d == EKV_ERR_INVALID || d == EKV_ERR_HIP, "demote pageable lo", 0);
  const ekv_status r = ekv_refine(&pool, 1, pairs, lens, bt, host, 2, 4, host, nullptr);
  expect(r == EKV_ERR_INVALID || r == EKV_ERR_HIP, "refine pageable lo", 0);
  const void* src[2] = {host, host + 65536 - 1};
  int32_t fresh[2] = {1, 1};
  expect(ekv_stage_blocks(&pool, 2, src, fresh, nullptr) == EKV_ERR_INVALID, "stage repeated block", 0);
  fresh[1] = 2;
  const ekv_status sb = ekv_stage_blocks(&pool, 2, src, fresh, nullptr);
  expect(sb == EKV_ERR_INVALID || sb == EKV_ERR_HIP, "stage pageable", 0);
  // the promotion protocol refuses a missing completion event before anything else
  expect(ekv_promote_begin(&pool, 2, src, fresh, nullptr, nullptr) == EKV_ERR_INVALID, "promote_begin no event", 0);
  expect(ekv_promote_publish(&pool, 1, pairs, fresh, bt, nullptr, 1, 4, nullptr, nullptr) == EKV_ERR_INVALID,
         "promote_publish no event", 0);
  expect(std::strlen(ekv_status_string(EKV_ERR_HOST)) > 0, "status string", 0);
  std::free(host);
  std::free(lens);
  std::free(bt);
  std::free(pairs);
}

}  // namespace

int main() {
  std::mt19937 rng(12345);
  lowering(rng);
  transitions(rng);
  controller(rng);
  arguments();
  if (failures) {
    std::fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  std::printf("host driver ok\n");
  return 0;
}
