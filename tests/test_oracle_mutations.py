"""The oracle's pins must catch plausible mistakes.  Each test plants one
mistake in the oracle (on the CPU, via monkeypatch) and checks that a pin
from the other test files fails."""

import numpy as np
import pytest

from oracle import attention, encoding, paged
from tests import test_oracle_attention as ta
from tests import test_oracle_encoding as te
from tests import test_oracle_transitions as tt


def test_rounding_instead_of_truncation_is_caught(monkeypatch, golden_dir):
    def rounded_hi(words):
        w = np.asarray(words, dtype=np.uint16).astype(np.uint32)
        return np.minimum((w + 0x80) >> 8, 0xFF).astype(np.uint8)
    monkeypatch.setattr(encoding, "hi_byte", rounded_hi)
    with pytest.raises(AssertionError):
        te.test_golden_words(golden_dir)
    with pytest.raises(AssertionError):
        te.test_refinement_is_exact_for_every_word()


def test_reading_the_wrong_pair_member_is_caught(monkeypatch):
    orig = encoding.base_word

    def member0_block_words(pool, bt_row, tag_row, i):
        phys = int(bt_row[i])
        if int(tag_row[i]) == paged.TARGET:
            return pool[phys].copy()
        return orig(paged.packed_bytes(pool, phys)[:, :, 0])
    monkeypatch.setattr(paged, "block_words", member0_block_words)
    with pytest.raises(AssertionError):
        ta.test_decode_matches_brute_force("bf16", 0.5)
    with pytest.raises(AssertionError):
        ta.test_prefill_with_base_prefix_matches_causal_sdpa_on_truncated_words()


def test_wrong_widening_is_caught(monkeypatch):
    def bad_widen(words, dtype):
        w = np.asarray(words, dtype=np.uint16)
        return (w.astype(np.uint32) << np.uint32(15)).view(np.float32).astype(np.float64)
    monkeypatch.setattr(encoding, "words_to_f64", bad_widen)
    with pytest.raises(AssertionError):
        ta.test_decode_matches_torch_sdpa(4)


def test_unnormalised_softmax_is_caught(monkeypatch):
    def bad(scores, values):
        return np.exp(scores - np.max(scores, axis=-1, keepdims=True)) @ values
    monkeypatch.setattr(attention, "_softmax_weighted", bad)
    with pytest.raises(AssertionError):
        ta.test_zero_query_gives_mean_of_values()


def test_dropped_low_byte_in_refine_is_caught(monkeypatch):
    monkeypatch.setattr(encoding, "refine_word",
                        lambda hi, lo: (np.asarray(hi, np.uint16) << np.uint16(8)).astype(np.uint16))
    with pytest.raises(AssertionError):
        tt.test_round_trip_restores_every_byte()


# ---- controller (Alg. 1) ---------------------------------------------------

from oracle import control as ocontrol
from tests import test_oracle_control as tc


@pytest.mark.parametrize("name,bad", [
    ("shortage", lambda demand, free: max(0, int(free) - int(demand))),           # sign
    ("demotion_count", lambda eligible, trigger, min_batch: min(eligible, trigger)),  # B_min dropped
    ("surplus", lambda demoted, delta: int(demoted)),                             # shortage not subtracted
    ("next_reserve", lambda reserve, decay, e: int(reserve) + int(e)),           # no decay
    ("promotion_budget", lambda free_post, reserve: int(free_post)),             # reserve ignored
])
def test_controller_formula_mistakes_are_caught(monkeypatch, name, bad):
    monkeypatch.setattr(ocontrol, name, bad)
    with pytest.raises(AssertionError):
        tc.test_hand_worked_trace()


def test_controller_rank_order_mistakes_are_caught(monkeypatch):
    orig = ocontrol.eligible_target_pairs
    monkeypatch.setattr(ocontrol, "eligible_target_pairs", lambda *a, **k: orig(*a, **k)[::-1])
    with pytest.raises(AssertionError):
        tc.test_hand_worked_trace()
    monkeypatch.undo()
    orig_b = ocontrol.eligible_base_pairs
    monkeypatch.setattr(ocontrol, "eligible_base_pairs", lambda *a, **k: orig_b(*a, **k)[::-1])
    with pytest.raises(AssertionError):
        tc.test_slack_limits_promotions()


def test_controller_ignoring_protected_pairs_is_caught(monkeypatch):
    def no_protection(tags, seq_lens, cfg, backed=None, page=16):
        plain = ocontrol.Config(min_batch=cfg.min_batch, decay=cfg.decay)
        return orig(tags, seq_lens, plain, backed, page)
    orig = ocontrol.eligible_target_pairs
    monkeypatch.setattr(ocontrol, "eligible_target_pairs", no_protection)
    with pytest.raises(AssertionError):
        tc.test_min_batch_capped_by_eligible_pairs()


# ---- 8-bit TARGET / 4-bit BASE ---------------------------------------------

from oracle import fp8 as ofp8
from tests import test_oracle_fp8 as tf


def test_fp8_swapped_nibble_order_is_caught(monkeypatch):
    monkeypatch.setattr(ofp8, "pack_nibbles",
                        lambda n: (np.asarray(n, np.uint8)[..., 1::2] | (np.asarray(n, np.uint8)[..., 0::2] << 4)
                                   ).astype(np.uint8))
    with pytest.raises(AssertionError):
        tf.test_nibble_packing_by_hand()


def test_fp8_low_nibble_as_base_is_caught(monkeypatch):
    monkeypatch.setattr(ofp8, "hi_nibble", lambda b: (np.asarray(b, np.uint8) & 0x0F).astype(np.uint8))
    with pytest.raises(AssertionError):
        tf.test_base_values_closed_form_and_exact_refinement()


def test_fp8_wrong_member_is_caught(monkeypatch):
    orig = ofp8.block_bytes

    def member0(pool, bt_row, tag_row, i):
        return orig(pool, bt_row, tag_row, i - (i % 2) if int(tag_row[i]) else i)
    monkeypatch.setattr(ofp8, "block_bytes", member0)
    with pytest.raises(AssertionError):
        tf.test_gather_matches_dense_copy_and_base_reads_packed_member()


# ---- metadata invariants ---------------------------------------------------

from oracle import validate as ov
from tests import test_oracle_validate as tv


def test_validate_member1_tag_decides_is_caught(monkeypatch):
    orig = ov.executed_as_base
    monkeypatch.setattr(ov, "executed_as_base",
                        lambda mode, by_range, b0, b1, j, t0, t1: orig(mode, by_range, b0, b1, j, t1, t0))
    with pytest.raises(AssertionError):
        tv.test_hand_built_batch_violations()


def test_validate_off_by_one_full_pair_is_caught(monkeypatch):
    monkeypatch.setattr(ov, "full_pair", lambda j, length, page: 2 * page * (j + 1) < length)
    with pytest.raises(AssertionError):
        tv.test_pairs_ending_at_the_length_are_full()


def test_validate_last_instead_of_first_index_is_caught(monkeypatch):
    def keep_last(self, kind, index):
        self.counts[kind] += 1
        self.first[kind] = index if self.first[kind] == ov.NONE else max(self.first[kind], index)
    monkeypatch.setattr(ov._Report, "flag", keep_last)
    with pytest.raises(AssertionError):
        tv.test_hand_built_batch_violations()


def test_fp8_append_mistakes_are_caught(monkeypatch):
    """Swapped K/V planes, or a slot split on the wrong page size, in the
    8-bit append fail its pins."""
    from oracle import fp8
    from tests import test_oracle_fp8 as tf

    def swapped(pool, slots, k_new, v_new):
        pool = np.array(pool, dtype=np.uint8, copy=True)
        page = pool.shape[3]
        for i, slot in enumerate(np.asarray(slots, dtype=np.int64)):
            pool[int(slot) // page, 1, :, int(slot) % page, :] = k_new[i]
            pool[int(slot) // page, 0, :, int(slot) % page, :] = v_new[i]
        return pool

    def wrong_split(pool, slots, k_new, v_new):
        pool = np.array(pool, dtype=np.uint8, copy=True)
        for i, slot in enumerate(np.asarray(slots, dtype=np.int64)):
            blk, off = divmod(int(slot), 8)
            blk %= pool.shape[0]
            pool[blk, 0, :, off, :] = k_new[i]
            pool[blk, 1, :, off, :] = v_new[i]
        return pool

    for bad in (swapped, wrong_split):
        monkeypatch.setattr(fp8, "append", bad)
        with pytest.raises(AssertionError):
            tf.test_append_places_rows_by_flat_index()
        with pytest.raises(AssertionError):
            tf.test_append_then_gather_reads_the_new_tokens()
