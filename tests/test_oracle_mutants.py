"""Planted-mistake checks: each plausible slip in the oracle (a dropped term,
a wrong index or sign, a transposed operand, a flipped tie rule) is compiled
into a mutant copy of the oracle module on the CPU, and at least one existing
pin test must fail against it. This shows the pins bite; the product path is
never involved."""
import importlib
import inspect
import sys
import types

import pytest

import oracle
import test_oracle_attention as TA
import test_oracle_compact_step as TC
import test_oracle_decode as TD
import test_oracle_geometry as TG
import test_oracle_lm_head as TL
import test_oracle_refresh as TR
import test_schedule as TS


def _mutant(modname: str, old: str, new: str):
    mod = importlib.import_module(modname)
    src = inspect.getsource(mod)
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    m = types.ModuleType(modname + "_mutant")
    m.__package__ = "oracle"
    m.__file__ = mod.__file__
    sys.modules[m.__name__] = m          # dataclasses resolve annotations through it
    exec(compile(src.replace(old, new), mod.__file__ + "[mutant]", "exec"), m.__dict__)
    return m


def _fails(fn, *args) -> bool:
    try:
        fn(*args)
    except Exception:
        return True
    return False


ATT = "oracle.attention"
DEC = "oracle.decode"
GAT = "oracle.gather"
GEO = "oracle.geometry"
CMP = "oracle.compact"
SCH = "oracle.schedule"
LMH = "oracle.lm_head"
RFR = "oracle.refresh"

MUTANTS = [
    # (module, anchor, replacement, exported name, pin tests that must catch it)
    (ATT, "scale = 1.0 / math.sqrt(D)", "scale = 1.0 / D", "dual_cache_block_attention",
     [(TA.test_matches_torch_sdpa_fp64, "f32")]),
    (ATT, "keys = np.concatenate([kpre, kblk, ksuf], axis=0)",
     "keys = np.concatenate([kpre, kblk, ksuf[:0]], axis=0)", "dual_cache_block_attention",
     [(TA.test_matches_torch_sdpa_fp64, "f32")]),
    (ATT, "kblk = widen(k_new[i, :t.B, c], dtype)",
     "kblk = widen(k_cache[t.row, c, t.off + t.s:t.off + t.e], dtype)", "dual_cache_block_attention",
     [(TA.test_matches_torch_sdpa_fp64, "f32")]),
    (ATT, "vblk = widen(v_new[i, :t.B, c], dtype)",
     "vblk = widen(v_cache[t.row, c, t.off + t.s:t.off + t.e], dtype)", "dual_cache_block_attention",
     [(TA.test_matches_torch_sdpa_fp64, "f32")]),
    (ATT, "for h in range(c * G, (c + 1) * G):", "for h in range(c, Hq, Hkv):",
     "dual_cache_block_attention", [(TA.test_gqa_equals_mha_with_repeated_kv_heads,),
                                    (TA.test_matches_scipy_softmax_with_gqa_and_padding,)]),
    (ATT, "w = w / w.sum(axis=1, keepdims=True)", "w = w / w.sum(axis=0, keepdims=True)",
     "dual_cache_block_attention", [(TA.test_matches_torch_sdpa_fp64, "f32")]),
    (ATT, "ksuf = widen(k_cache[t.row, c, t.off + t.e:t.off + t.len], dtype)",
     "ksuf = widen(k_cache[t.row, c, t.e:t.len], dtype)", "dual_cache_block_attention",
     [(TA.test_matches_scipy_softmax_with_gqa_and_padding,)]),
    (ATT, "kc_out[t.row, c, t.off + t.s:t.off + t.e] = k_new[i, :t.B, c]",
     "kc_out[t.row, c, t.s:t.e] = k_new[i, :t.B, c]", "dual_cache_block_attention",
     [(TA.test_write_back_touches_only_block_cells,)]),
    (DEC, "if conf[i, j] >= tau", "if conf[i, j] > tau", "parallel_decode",
     [(TD.test_at_threshold_is_inclusive,)]),
    (DEC, "a = int(np.argmax(x))", "a = int(len(x) - 1 - np.argmax(x[::-1]))", "parallel_decode",
     [(TD.test_argmax_tie_goes_to_smallest_id,)]),
    (DEC, "key=lambda j: (-conf[i, j], j)", "key=lambda j: (-conf[i, j], -j)", "parallel_decode",
     [(TD.test_uniform_logits_unmask_one_at_smallest_masked_position,)]),
    (DEC, "max(int(q_min), sum(", "min(int(q_min), sum(", "parallel_decode",
     [(TD.test_fixed_quota_variant,)]),
    (DEC, "c = 1.0 / np.exp(x - mx).sum()", "c = 1.0 / np.exp(x - mx)[1:].sum()", "parallel_decode",
     [(TD.test_single_spike_closed_form,)]),
    (DEC, "done[i] = 1 if n_sel == len(M) else 0", "done[i] = 1 if n_sel >= 1 else 0", "parallel_decode",
     [(TD.test_uniform_logits_unmask_one_at_smallest_masked_position,)]),
    (GAT, "out[i, j] = dense[q.row, q.off + q.s + j]", "out[i, j] = dense[q.row, q.off + q.p + j]",
     "gather_active_blocks", [(TG.test_gather_reads_hand_enumerated_cells,)]),
    (GAT, "pos[i, j] = q.s + j", "pos[i, j] = q.off + q.s + j", "gather_active_blocks",
     [(TG.test_gather_reads_hand_enumerated_cells,)]),
    (GAT, "out[q.row, q.off + q.s + j] = compact[i, j]", "out[q.row, q.off + q.s + j - 1] = compact[i, j]",
     "scatter_active_blocks", [(TG.test_gather_scatter_identities,)]),
    (GEO, "K = math.ceil(g / L)", "K = g // L", "geometry", [(TG.test_partial_last_block,)]),
    (GEO, "B = min(L, g - k * L)", "B = L", "geometry", [(TG.test_partial_last_block,)]),
    (GEO, "s = p + k * L", "s = p + (k + 1) * L", "geometry",
     [(TG.test_tiny_geometry_matches_hand_enumeration,)]),
    (GEO, "return len(reqs) * max(int(r[\"p\"]) + (int(r[\"k\"]) + 1) * L for r in reqs)",
     "return len(reqs) * max(int(r[\"p\"]) + int(r[\"k\"]) * L for r in reqs)", "bbox_cost",
     [(TG.test_tiny_geometry_matches_hand_enumeration,)]),
    (CMP, "out_k[l, dr, h, dc:dc + ln] = sk[l, sr, h, sc:sc + ln]",
     "out_k[l, dr, h, dc:dc + ln] = sk[l, dr, h, sc:sc + ln]", "kv_scatter_compact",
     [(TC.test_stable_slot_plan_leaves_survivors_untouched,)]),
    (SCH, "return self.p + (self.b + 1) * self.L", "return self.p + self.b * self.L", "schedule",
     [(TS.test_eq1_cost_matches_bounding_box_definition,), (TS.test_fig1_example2_bounding_box_shrink_expands_the_batch,)]),
    (SCH, "if c.p + self.L <= box and cost(self.active, c) <= self.budget:",
     "if False and c.p + self.L <= box and cost(self.active, c) <= self.budget:", "schedule",
     [(TS.test_admission_postconditions_and_completion, 2)]),
    (SCH, "if r.b >= r.K or r.id in eos:", "if r.b >= r.K:", "schedule",
     [(TS.test_eos_evicts_at_the_block_boundary,)]),
    (SCH, "len(self.active) < self.fixed_batch", "len(self.active) <= self.fixed_batch", "schedule",
     [(TS.test_fig1_example1_eviction_and_refill,)]),
    (LMH, "out[:, v0:v0 + chunk] = h @ widen(w_vocab[v0:v0 + chunk], dtype).T",
     "out[:, v0:v0 + chunk] = h[:, 1:] @ widen(w_vocab[v0:v0 + chunk], dtype)[:, 1:].T", "lm_head_decode",
     [(TL.test_matches_brute_force_products, 0, 3)]),
    (LMH, "rows = {key: lg[a] for a, key in enumerate(keys)}",
     "rows = {key: lg[min(a + 1, len(keys) - 1)] for a, key in enumerate(keys)}", "lm_head_decode",
     [(TL.test_matches_brute_force_products, 1, 4096)]),
    (LMH, "out[:, v0:v0 + chunk] = h @ widen(w_vocab[v0:v0 + chunk], dtype).T",
     "out[:, v0:v0 + chunk] = h @ widen(w_vocab[v0:v0 + chunk][::-1], dtype).T", "lm_head_decode",
     [(TL.test_identity_head_gives_softmax_of_the_hidden_state,)]),
    (RFR, "x1 * c - x2 * s", "x1 * c + x2 * s", "rope", [(TR.test_rope_two_features_is_a_plane_rotation,)]),
    (RFR, "x1, x2 = x[..., :half], x[..., half:]", "x1, x2 = x[..., 0::2], x[..., 1::2]", "rope",
     [(TR.test_rope_pairs_feature_f_with_f_plus_half,)]),
    (RFR, "inv_freq = float(base) ** (-2.0 * f / D)", "inv_freq = float(base) ** (-1.0 * f / D)", "rope",
     [(TR.test_rope_pairs_feature_f_with_f_plus_half,), (TR.test_rope_equals_complex_multiplication,)]),
    (RFR, "return position_ids(mask)[off:off + ln]", "return np.arange(off, off + ln)", "dual_cache_refresh",
     [(TR.test_placement_in_the_box_does_not_matter,)]),
    (RFR, "qr = rope(widen(q_row[off:off + ln], dtype), pos[:, None], rope_base)",
     "qr = widen(q_row[off:off + ln], dtype)", "dual_cache_refresh",
     [(TR.test_block_rows_match_block_attention_on_the_refreshed_cache,)]),
    (RFR, "vv = widen(v_row[off:off + ln], dtype)",
     "vv = rope(widen(v_row[off:off + ln], dtype), pos[:, None], rope_base)", "dual_cache_refresh",
     [(TR.test_uniform_values_and_one_token_row,)]),
    (RFR, "kc[row, c, off:off + ln] = kr[:, c]", "kc[row, c, off:off + ln] = widen(k[row, off:off + ln, c], dtype)",
     "dual_cache_refresh", [(TR.test_block_rows_match_block_attention_on_the_refreshed_cache,)]),
    (RFR, "c = h // G", "c = h % Hkv", "dual_cache_refresh", [(TR.test_unrotated_refresh_matches_torch_sdpa, "f32")]),
    (RFR, "scale = 1.0 / math.sqrt(D)", "scale = 1.0 / D", "dual_cache_refresh",
     [(TR.test_unrotated_refresh_matches_torch_sdpa, "f32")]),
    (RFR, "kr = rope(widen(k_row[off:off + ln], dtype)", "kr = rope(widen(k_row[off + 1:off + ln + 1], dtype)",
     "dual_cache_refresh", [(TR.test_unrotated_refresh_matches_torch_sdpa, "f32")]),
]


@pytest.mark.parametrize("modname,old,new,name,pins", MUTANTS,
                         ids=[f"{m[0].split('.')[1]}:{m[2][:40]}" for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, modname, old, new, name, pins):
    # sanity: every pin passes on the real oracle
    for pin in pins:
        assert not _fails(pin[0], *pin[1:]), f"{pin[0].__name__} fails on the real oracle"
    m = _mutant(modname, old, new)
    if modname == SCH:                   # the scheduler pins use the module itself
        monkeypatch.setattr(TS, "osch", m)
    else:
        monkeypatch.setattr(oracle, name, getattr(m, name))
    assert any(_fails(pin[0], *pin[1:]) for pin in pins), "no pin caught the planted mistake"
