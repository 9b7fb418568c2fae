"""Pressure-aware fidelity control (oracle).

TEST INFRASTRUCTURE ONLY (see the package docstring).

§3.3, Alg. 1 and App. B.1: once per scheduling step the controller

1. probes the block demand D_t of the step and forms the shortage
   Delta_t = max(0, D_t - F_t) against the free blocks F_t (the probe is
   skipped, Delta_t = 0, while F_t exceeds the static guard A_max);
2. if Delta_t > 0, takes the eligible TARGET pairs P_d, demotes
   n_d = min(|P_d|, max(Delta_t, B_min)) of them in rank order, and records
   the surplus E_t = max(0, n_d - Delta_t) (each demoted pair frees one
   block); otherwise E_t = 0;
3. after the step's required scheduling, with F_post free blocks left,
   updates the decaying reserve R_t = max(0, R_{t-1} - lambda) + E_t and the
   promotion budget P_t = max(0, F_post - R_t), and, if P_t > 0 and the
   transfer path has slack, promotes eligible BASE pairs (one block each).

App. C.7 (ablation settings) adds three switches: a free-capacity watermark in place
of the shortage trigger, eager promotion (no reserve in the budget) and no
promotion at all.

Readings where the paper is silent (each listed in the design notes):

* eligible TARGET pair (s, j): both members TARGET and full
  (32 (j + 1) <= L_s), outside the protected sink (j >= sink_pairs) and
  recent window (j < L_s // 32 - recent_pairs), and backed (if a backing
  mask is given, its entry for member 0);
* rank_and_batch: oldest first -- ascending (j, s) -- so that every
  sequence's BASE pairs stay one run right after its sink;
* eligible BASE pairs are promoted newest first -- descending j, then
  ascending s -- which shrinks that run from its recent end;
* the number of promotions is min(P_t, slack, eligible BASE pairs), slack
  being the pairs the transfer path can take this step;
* watermark policy: triggered while F_t < W, demoting
  min(|P_d|, max(W - F_t, B_min)); the surplus is still measured against
  the step's shortage max(0, D_t - F_t);
* eager promotion: P_t = F_post (the reserve is still kept, unused).

Pair lists are int32 arrays of shape [n, 2] holding (s, j).
"""

import numpy as np

SHORTAGE = 0
WATERMARK = 1


class Config:
    def __init__(self, min_batch=16, decay=2, a_max=-1, sink_pairs=0, recent_pairs=0, policy=SHORTAGE,
                 watermark=0, eager=False, no_promotion=False):
        self.min_batch = int(min_batch)     # B_min^d (App. B.1 default 16)
        self.decay = int(decay)             # lambda (App. B.1 default 2)
        self.a_max = int(a_max)             # A_max; negative: always probe
        self.sink_pairs = int(sink_pairs)
        self.recent_pairs = int(recent_pairs)
        self.policy = policy
        self.watermark = int(watermark)
        self.eager = bool(eager)
        self.no_promotion = bool(no_promotion)


def eligible_target_pairs(tags, seq_lens, cfg, backed=None, page=16):
    """P_d in rank order (ascending j, then s)."""
    out = []
    for s, length in enumerate(seq_lens):
        full_pairs = int(length) // (2 * page)
        for j in range(cfg.sink_pairs, full_pairs - cfg.recent_pairs):
            if tags[s, 2 * j] != 0 or tags[s, 2 * j + 1] != 0:
                continue
            if backed is not None and backed[s, 2 * j] == 0:
                continue
            out.append((j, s))
    out.sort()
    return np.array([(s, j) for j, s in out], dtype=np.int32).reshape(-1, 2)


def eligible_base_pairs(tags, seq_lens, page=16):
    """BASE pairs in promotion order (descending j, then ascending s)."""
    out = []
    for s, length in enumerate(seq_lens):
        nblk = -(-int(length) // page)
        for j in range(nblk // 2):
            if tags[s, 2 * j] != 0 and tags[s, 2 * j + 1] != 0:
                out.append((-j, s))
    out.sort()
    return np.array([(s, -mj) for mj, s in out], dtype=np.int32).reshape(-1, 2)


def shortage(demand, free):
    """Delta_t = max(0, D_t - F_t)."""
    return max(0, int(demand) - int(free))


def demotion_count(eligible, trigger, min_batch):
    """n_d = min(|P_d|, max(Delta_t, B_min))."""
    return min(int(eligible), max(int(trigger), int(min_batch)))


def surplus(demoted, delta):
    """E_t = max(0, |B_d| - Delta_t)."""
    return max(0, int(demoted) - int(delta))


def next_reserve(reserve, decay, surplus_t):
    """R_t = max(0, R_{t-1} - lambda) + E_t."""
    return max(0, int(reserve) - int(decay)) + int(surplus_t)


def promotion_budget(free_post, reserve):
    """P_t = max(0, F_post - R_t)."""
    return max(0, int(free_post) - int(reserve))


class Controller:
    """Alg. 1 over a host view of the pool; the caller applies the lists."""

    def __init__(self, cfg):
        self.cfg = cfg
        self.reserve = 0     # R_{t-1}
        self.surplus = 0     # E_t of the current step
        self.shortage = 0    # Delta_t of the current step
        self.budget = 0      # P_t of the current step

    def demotion(self, demand, free, tags, seq_lens, backed=None, page=16):
        """First half of a step: returns B_d (pairs to demote now)."""
        cfg = self.cfg
        if cfg.a_max >= 0 and free > cfg.a_max:
            delta = 0                                    # probe skipped
        else:
            delta = shortage(demand, free)
        trigger = max(0, cfg.watermark - int(free)) if cfg.policy == WATERMARK else delta
        self.shortage = delta
        self.surplus = 0
        if trigger == 0:
            return np.zeros((0, 2), dtype=np.int32)
        cand = eligible_target_pairs(tags, seq_lens, cfg, backed, page)
        chosen = cand[:demotion_count(len(cand), trigger, cfg.min_batch)]
        self.surplus = surplus(len(chosen), delta)
        return chosen

    def promotion(self, free_post, slack, tags, seq_lens, page=16):
        """Second half, after required scheduling: returns B_p (pairs to
        promote, one free block each)."""
        cfg = self.cfg
        self.reserve = next_reserve(self.reserve, cfg.decay, self.surplus)
        self.budget = promotion_budget(free_post, 0 if cfg.eager else self.reserve)
        if cfg.no_promotion or self.budget <= 0 or slack <= 0:
            return np.zeros((0, 2), dtype=np.int32)
        cand = eligible_base_pairs(tags, seq_lens, page)
        return cand[:min(self.budget, int(slack))]
