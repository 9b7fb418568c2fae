// Pressure-aware fidelity control (paper §3.3, Alg. 1; App. B.1; the
// ablation switches of App. C.7), host only.  Declarations and contracts:
// include/ekv.h.
//
// One scheduling step is two calls around the serving scheduler:
//   ekv_ctrl_demotion   before scheduling: shortage Delta_t = max(0, D_t -
//                       F_t) (no probe while F_t > A_max); if positive,
//                       n_d = min(|P_d|, max(Delta_t, B_min)) eligible
//                       TARGET pairs in rank order; surplus
//                       E_t = max(0, n_d - Delta_t).
//   ekv_ctrl_promotion  after scheduling, with F_post free blocks:
//                       R_t = max(0, R_{t-1} - lambda) + E_t,
//                       P_t = max(0, F_post - R_t), and up to
//                       min(P_t, slack) eligible BASE pairs.
// Rank orders (the paper leaves the signals open): demotion takes the
// oldest unprotected TARGET pairs first -- ascending (pair index, sequence)
// -- and promotion the newest BASE pairs first -- descending pair index,
// then ascending sequence -- so every sequence's BASE pairs stay one run
// next to its protected sink and lowering stays structured.
#include <algorithm>

#include "ekv.h"
#include "host_status.h"

namespace {

using ekv::fail;

ekv_status check_view(const char* who, const uint8_t* tags, const int32_t* lens, int32_t batch,
                      int32_t max_blocks, int32_t page, const int32_t* out, const int32_t* n_out) {
  if (batch < 0 || max_blocks <= 0 || page <= 0) return fail(EKV_ERR_INVALID, "%s: bad sizes", who);
  if (!n_out || (batch > 0 && (!tags || !lens || !out))) return fail(EKV_ERR_INVALID, "%s: NULL array", who);
  for (int s = 0; s < batch; ++s)
    if (lens[s] < 0 || (long long)lens[s] > (long long)max_blocks * page)
      return fail(EKV_ERR_INVALID, "%s: sequence %d length %d out of range", who, s, lens[s]);
  return EKV_OK;
}

ekv_status check_config(const char* who, const ekv_ctrl_config* c, const ekv_ctrl_state* st) {
  if (!c || !st) return fail(EKV_ERR_INVALID, "%s: NULL config or state", who);
  if (c->min_batch < 0 || c->decay < 0 || c->sink_pairs < 0 || c->recent_pairs < 0 || c->watermark < 0)
    return fail(EKV_ERR_INVALID, "%s: negative parameter", who);
  if (c->policy != EKV_CTRL_SHORTAGE && c->policy != EKV_CTRL_WATERMARK)
    return fail(EKV_ERR_INVALID, "%s: unknown policy %d", who, c->policy);
  if (c->flags & ~(EKV_CTRL_EAGER_PROMOTION | EKV_CTRL_NO_PROMOTION))
    return fail(EKV_ERR_INVALID, "%s: unknown flags 0x%x", who, c->flags);
  if (st->reserve < 0) return fail(EKV_ERR_INVALID, "%s: negative reserve", who);
  return EKV_OK;
}

}  // namespace

extern "C" {

ekv_status ekv_ctrl_demotion(const ekv_ctrl_config* cfg, ekv_ctrl_state* st, int32_t demand,
                             int32_t free_blocks, const uint8_t* h_tags, const int32_t* h_seq_lens,
                             const uint8_t* h_backed, int32_t batch, int32_t max_blocks,
                             int32_t page_size, int32_t* h_pairs_out, int32_t max_pairs, int32_t* n_out) {
  return ekv::guard("ekv_ctrl_demotion", [&]() -> ekv_status {
    ekv_status e = check_config("ekv_ctrl_demotion", cfg, st);
    if (e != EKV_OK) return e;
    if ((e = check_view("ekv_ctrl_demotion", h_tags, h_seq_lens, batch, max_blocks, page_size, h_pairs_out,
                        n_out)) != EKV_OK)
      return e;
    if (demand < 0 || free_blocks < 0 || max_pairs < 0)
      return fail(EKV_ERR_INVALID, "ekv_ctrl_demotion: negative demand, free count or capacity");
    *n_out = 0;
    // Delta_t: the demand probe runs only while free capacity is at or below A_max
    const int delta = (cfg->a_max >= 0 && free_blocks > cfg->a_max) ? 0 : std::max(0, demand - free_blocks);
    const int trigger = cfg->policy == EKV_CTRL_WATERMARK ? std::max(0, cfg->watermark - free_blocks) : delta;
    if (trigger == 0) {
      st->shortage = delta;
      st->surplus = 0;
      return EKV_OK;
    }
    const int want = std::max(trigger, cfg->min_batch);   // n_d before the cap by |P_d|
    // eligible pairs of sequence s: sink_pairs <= j < len/32 - recent_pairs, TARGET, backed
    int jmax = 0;
    for (int s = 0; s < batch; ++s) jmax = std::max(jmax, h_seq_lens[s] / (2 * page_size) - cfg->recent_pairs);
    int n = 0;
    for (int j = cfg->sink_pairs; j < jmax && n < want; ++j) {
      for (int s = 0; s < batch && n < want; ++s) {
        if (j >= h_seq_lens[s] / (2 * page_size) - cfg->recent_pairs) continue;
        const uint8_t* row = h_tags + (size_t)s * max_blocks;
        if (row[2 * j] != 0 || row[2 * j + 1] != 0) continue;
        if (h_backed && h_backed[(size_t)s * max_blocks + 2 * j] == 0) continue;
        if (n == max_pairs) return fail(EKV_ERR_INVALID, "ekv_ctrl_demotion: more than %d pairs chosen", max_pairs);
        h_pairs_out[2 * n] = s;
        h_pairs_out[2 * n + 1] = j;
        ++n;
      }
    }
    *n_out = n;
    st->shortage = delta;
    st->surplus = std::max(0, n - delta);
    return EKV_OK;
  });
}

ekv_status ekv_ctrl_promotion(const ekv_ctrl_config* cfg, ekv_ctrl_state* st, int32_t free_post, int32_t slack,
                              const uint8_t* h_tags, const int32_t* h_seq_lens, int32_t batch,
                              int32_t max_blocks, int32_t page_size, int32_t* h_pairs_out, int32_t max_pairs,
                              int32_t* n_out) {
  return ekv::guard("ekv_ctrl_promotion", [&]() -> ekv_status {
    ekv_status e = check_config("ekv_ctrl_promotion", cfg, st);
    if (e != EKV_OK) return e;
    if ((e = check_view("ekv_ctrl_promotion", h_tags, h_seq_lens, batch, max_blocks, page_size, h_pairs_out,
                        n_out)) != EKV_OK)
      return e;
    if (free_post < 0 || slack < 0 || max_pairs < 0)
      return fail(EKV_ERR_INVALID, "ekv_ctrl_promotion: negative free count, slack or capacity");
    *n_out = 0;
    st->reserve = std::max(0, st->reserve - cfg->decay) + st->surplus;   // R_t
    const int protect = (cfg->flags & EKV_CTRL_EAGER_PROMOTION) ? 0 : st->reserve;
    st->budget = std::max(0, free_post - protect);                     // P_t
    if ((cfg->flags & EKV_CTRL_NO_PROMOTION) || st->budget == 0 || slack == 0) return EKV_OK;
    const int want = std::min(st->budget, slack);
    int jtop = -1;   // highest pair index whose two blocks hold tokens
    for (int s = 0; s < batch; ++s) jtop = std::max(jtop, (h_seq_lens[s] + page_size - 1) / page_size / 2 - 1);
    int n = 0;
    for (int j = jtop; j >= 0 && n < want; --j) {
      for (int s = 0; s < batch && n < want; ++s) {
        if (2 * j + 1 >= (h_seq_lens[s] + page_size - 1) / page_size) continue;
        const uint8_t* row = h_tags + (size_t)s * max_blocks;
        if (row[2 * j] == 0 || row[2 * j + 1] == 0) continue;
        if (n == max_pairs) return fail(EKV_ERR_INVALID, "ekv_ctrl_promotion: more than %d pairs chosen", max_pairs);
        h_pairs_out[2 * n] = s;
        h_pairs_out[2 * n + 1] = j;
        ++n;
      }
    }
    *n_out = n;
    return EKV_OK;
  });
}

}  // extern "C"
