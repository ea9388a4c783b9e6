"""Plant plausible mistakes in copies of the oracle (CPU only) and require that
the pins catch every one of them: a dropped term, a wrong comparison, a wrong
operand or index must fail at least one check."""
import sys
import types

import pytest

from oracle import layercheck_oracle as O
from tests import oracle_pins as P
from tests import test_oracle_adamw as A
from tests import test_oracle_sgd as G
from tests.test_bruteforce_tiny import run_bruteforce

SRC = open(O.__file__).read()

MUTANTS = {
    "denominator_uses_current": ("B += float(np.sum(np.abs(y)))", "B += float(np.sum(np.abs(x)))"),
    "widen_bf16_as_fp16": ("return (values.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)",
                           "return values.view(np.float16).astype(np.float64)"),
    "widen_drops_low_byte": ("return (values.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)",
                             "return ((values.astype(np.uint32) & np.uint32(0xFF00)) << np.uint32(16)).view(np.float32).astype(np.float64)"),
    "signed_difference": ("A += float(np.sum(np.abs(x - y)))", "A += float(np.sum(x - y))"),
    "eps_dropped": ("np.float64(B / n + eps_w)", "np.float64(B / n)"),
    "eps_outside_mean": ("np.float64(B / n + eps_w)", "np.float64((B + eps_w) / n)"),
    "per_tensor_count": ("n += int(w.size)", "n = int(w.size)"),
    "strict_threshold": ("by_drift = delta[l] >= K", "by_drift = delta[l] > K"),
    "strict_staleness": ("by_age = age >= s_max", "by_age = age > s_max"),
    "lr_scale_ignored": ("K = k0[l] * lr_scale", "K = k0[l]"),
    "lr_scale_inverted": ("K = k0[l] * lr_scale", "K = k0[l] / lr_scale"),
    "no_reset": ("            if mask[l]:  # Eq. 4: reset on persist\n                self.delta[l] = 0.0\n",
                 "            if mask[l]:  # Eq. 4: reset on persist\n"),
    "no_timestamp": ("                self.delta[l] = 0.0\n                self.t_last[l] = step\n        self.scored_step = None",
                     "                self.delta[l] = 0.0\n        self.scored_step = None"),
    "accum_overwrites": ("            if self.mode == MODE_ACCUM:\n                self.delta[l] = self.delta[l] + u",
                         "            if self.mode == MODE_ACCUM:\n                self.delta[l] = u"),
    "adamw_accum_overwrites": ("            self.u[l] = u\n            self.delta[l] = self.delta[l] + u",
                               "            self.u[l] = u\n            self.delta[l] = u"),
    "accum_shadow_stale": ("        if self.mode == MODE_ACCUM:\n            # the next step's",
                           "        if False:\n            # the next step's"),
    "forced_count_wrong": ("forced[l] = 0 if by_drift else 1", "forced[l] = 1 if by_age else 0"),
    "pack_descending_ids": ("sel = [l for l in range(self.N) if self.mask[l]]\n        if first_rank < 0",
                            "sel = [l for l in reversed(range(self.N)) if self.mask[l]]\n        if first_rank < 0"),
    "snapshot_pack_keeps_shadow": ("        if self.mode == MODE_SNAPSHOT:\n            for l in sel[first_rank:last]:",
                                   "        if False:\n            for l in sel[first_rank:last]:"),
    "restore_keeps_delta": ("            self.delta[l] = 0.0\n            self.t_last[l] = int(v[\"step\"])",
                            "            self.t_last[l] = int(v[\"step\"])"),
    "restore_stamps_t_fail": ("            self.t_last[l] = int(v[\"step\"])\n            chosen[l]",
                              "            self.t_last[l] = t_fail\n            chosen[l]"),
    "sums_not_means": ("np.float64(A / n) / np.float64(B / n + eps_w)", "np.float64(A) / np.float64(B + eps_w)"),
    "master_after_moments": ('return (["weight"] + (["master"] if has_master else [])\n            + (["exp_avg", "exp_avg_sq"] if has_moments else []))',
                             'return (["weight"] + (["exp_avg", "exp_avg_sq"] if has_moments else [])\n            + (["master"] if has_master else []))'),
    "snapshot_score_refreshes_shadow": ("        if self.mode == MODE_ACCUM:\n            # the next step's W(t-1)",
                                        "        if True:\n            # the next step's W(t-1)"),
    "adamw_betas_swapped": ('m_new = (sc["b1"] * m).astype(f) + (sc["omb1"] * g).astype(f)',
                            'm_new = (sc["b2"] * m).astype(f) + (sc["omb2"] * g).astype(f)'),
    "adamw_v_linear_in_g": ('(sc["omb2"] * (g * g).astype(f)).astype(f)', '(sc["omb2"] * np.abs(g)).astype(f)'),
    "no_padding": ("out += bytes(padded(len(raw)) - len(raw))", "pass"),
    "moments_swapped": ('["exp_avg", "exp_avg_sq"] if has_moments', '["exp_avg_sq", "exp_avg"] if has_moments'),
    "restore_oldest": ('if best is None or v["step"] > best_step:', 'if best is None or v["step"] < best_step:'),
    "restore_ignores_t_fail": ('if v["step"] <= t_fail and v["mask"][l]:', 'if v["mask"][l]:'),
    "restore_offset_counts_all": ('off = sum(self.R[j] for j in range(l) if v["mask"][j])',
                                  'off = sum(self.R[j] for j in range(l))'),
    "restore_keeps_old_shadow": ("            for s in self.by_layer[l]:\n                s.shadow[...] = s.weight\n            self.delta[l] = 0.0",
                                 "            self.delta[l] = 0.0"),
    "stats_ages_before_reset": ("ages = [step - self.t_last[l] for l in range(self.N)]",
                                "ages = [step - self._pre_t_last[l] for l in range(self.N)]"),
    "payload_counts_every_layer": ('"payload_bytes": sum(self.R[l] for l in range(self.N) if mask[l]),',
                                   '"payload_bytes": sum(self.R),'),
    "score_allows_repeat_step": ("    def score(self, step: int) -> None:\n        if step <= self.last_step:",
                                 "    def score(self, step: int) -> None:\n        if step < self.last_step:"),
    "restore_keeps_last_step": ("        self.last_step = t_fail\n        self.scored_step = None\n        self.mask = None",
                                "        self.scored_step = None\n        self.mask = None"),
    "select_accepts_bad_lr_scale": ('        if not (lr_scale > 0.0) or lr_scale == float("inf"):', "        if False:"),
    "pack_first_rank_unchecked": ('        if first_rank < 0 or first_rank > len(sel):\n            raise OracleError(LC_ERR_INVALID_ARG, "first_rank out of range")\n', ""),
    "record_moments_when_absent": ('            + (["exp_avg", "exp_avg_sq"] if has_moments else []))',
                                   '            + ["exp_avg", "exp_avg_sq"])'),
    "fused_step_in_snapshot": ('        if self.mode != MODE_ACCUM:\n            raise OracleError(LC_ERR_BAD_STATE, "the fused optimizer step accumulates (ACCUM mode)")\n', ''),
    "fused_step_not_selectable": ('        self.last_step = step\n        self.scored_step = step\n        self.unpacked = set()\n        self.mask = None\n\n    def adamw_step_score',
                                  '        self.last_step = step\n        self.unpacked = set()\n        self.mask = None\n\n    def adamw_step_score'),
    "sgd_decay_scales_the_step": ('    return (p1 - (sc["lr"] * g.astype(f)).astype(f)).astype(f)',
                                  '    return (p1 - (sc["lr"] * sc["decay"] * g.astype(f)).astype(f)).astype(f)'),
    "init_accepts_unordered_layers": ("if not (0 <= s.layer < n_layers) or s.layer < last or s.numel == 0:",
                                      "if not (0 <= s.layer < n_layers) or s.numel == 0:"),
    "init_accepts_master_mismatch": ('            if (s.master is None) == has_master:\n                raise OracleError(LC_ERR_INVALID_ARG, "master presence mismatch")\n', ""),
    "init_accepts_smax_zero": ("if len(k0) != n_layers or s_max < 1 or not (eps_w >= 0.0)",
                               "if len(k0) != n_layers or s_max < 0 or not (eps_w >= 0.0)"),
    "init_accepts_negative_eps": ("or not (eps_w >= 0.0) or eps_w", "or eps_w"),
    "init_accepts_infinite_eps": ('or not (eps_w >= 0.0) or eps_w == float("inf"):', "or not (eps_w >= 0.0):"),
    "init_accepts_missing_layer": ('        if any(len(g) == 0 for g in self.by_layer):\n            raise OracleError(LC_ERR_INVALID_ARG, "layer without tensors")\n', ""),
    "snapshot_pack_refreshes_unpacked": ("            for l in sel[first_rank:last]:\n                for s in self.by_layer[l]:\n                    s.shadow[...] = s.weight",
                                         "            for l in sel:\n                for s in self.by_layer[l]:\n                    s.shadow[...] = s.weight"),
    "init_accepts_negative_k0": ("        if not all(k >= 0.0 for k in k0):  # refuses NaN too", "        if False:"),
    "plan_skips_mask_length": ('            if m.shape != (self.N,):\n                raise OracleError(LC_ERR_INVALID_ARG, "mask length")\n', ''),
    "pack_without_selection": ('        if self.mask is None:\n            raise OracleError(LC_ERR_BAD_STATE, "nothing selected")\n', ''),
    "restore_leaves_a_score": ("        self.last_step = t_fail\n        self.scored_step = None", "        self.last_step = t_fail\n        self.scored_step = t_fail"),
    "select_twice_per_score": ("        self.scored_step = None\n        self.mask = mask\n        self.mask_step = step", "        self.mask = mask\n        self.mask_step = step"),
    "delta_accumulated_in_fp32": ("            if self.mode == MODE_ACCUM:\n                self.delta[l] = self.delta[l] + u",
                                  "            if self.mode == MODE_ACCUM:\n                self.delta[l] = float(np.float32(self.delta[l] + u))"),
    "restore_keeps_pending_selection": ("        self.mask = None\n        self.unpacked = set()\n        return chosen",
                                        "        self.mask = None\n        return chosen"),
    "adamw_eps_squared": ('    denom = (np.sqrt(v_hat).astype(f) + sc["eps"]).astype(f)',
                          '    denom = (np.sqrt(v_hat).astype(f) + sc["eps"] * sc["eps"]).astype(f)'),
    "age_off_by_one": ("age = step - t_last[l]", "age = step - t_last[l] - 1"),
    "plan_allows_duplicate_steps": ('        if dup:\n            raise OracleError(LC_ERR_INVALID_ARG, f"layer {l}: two versions at step {best_step}")\n', ""),
    "plan_falls_back_silently": ('        if best is None:\n            raise OracleError(LC_ERR_NO_VERSION, f"layer {l}: no persisted version <= {t_fail}")\n',
                                 "        if best is None:\n            best = 0\n"),
    "capacity_error_dropped": ('        if last == first_rank and first_rank < len(sel):\n            raise OracleError(LC_ERR_CAPACITY, "record does not fit")\n', ""),
    "record_segments_reversed": ("            for s in g:\n                raw = getattr(s, arr).tobytes()",
                                 "            for s in reversed(g):\n                raw = getattr(s, arr).tobytes()"),
    "restore_segments_reversed": ("                for s in self.by_layer[l]:\n                    dst = getattr(s, arr)",
                                  "                for s in reversed(self.by_layer[l]):\n                    dst = getattr(s, arr)"),
    "plan_skips_payload_check": ('            if len(v["payload"]) != need:\n                raise OracleError(LC_ERR_INVALID_ARG, "payload size does not match mask")\n', ""),
    "restore_reads_unpadded": ("                    pos += padded(nb)", "                    pos += nb"),
    "adamw_bias_step_off_by_one": ('"c1": f(1.0 / (1.0 - beta1 ** t)), "c2": f(1.0 / (1.0 - beta2 ** t)),',
                                   '"c1": f(1.0 / (1.0 - beta1 ** (t + 1))), "c2": f(1.0 / (1.0 - beta2 ** (t + 1))),'),
    "adamw_decay_after_update": ('    p1 = (p * sc["decay"]).astype(f) if decayed else p.astype(f)\n    p_new = (p1 - (sc["lr"] * upd).astype(f)).astype(f)',
                                 '    p_new = (p - (sc["lr"] * upd).astype(f)).astype(f)\n    p_new = (p_new * sc["decay"]).astype(f) if decayed else p_new'),
    "adamw_m_hat_from_old_m": ('    m_hat = (m_new * sc["c1"]).astype(f)', '    m_hat = (m * sc["c1"]).astype(f)'),
    "adamw_c2_uses_beta1": ('"c2": f(1.0 / (1.0 - beta2 ** t)),', '"c2": f(1.0 / (1.0 - beta1 ** t)),'),
    "optim_reads_weights_not_master": ("            if s.master is not None:\n                p_old = s.master.copy()",
                                       "            if False:\n                p_old = s.master.copy()"),
    "optim_master_not_written": ("            if s.master is not None:\n                s.master[...] = p_new",
                                 "            if False:\n                s.master[...] = p_new"),
    "optim_drift_without_eps": ("_, _, _, u = layer_update_score([s._p_new for s in g], [s._p_old for s in g], DT_F32, self.eps_w)",
                                "_, _, _, u = layer_update_score([s._p_new for s in g], [s._p_old for s in g], DT_F32, 0.0)"),
    "optim_drift_on_stored_weights": ("_, _, _, u = layer_update_score([s._p_new for s in g], [s._p_old for s in g], DT_F32, self.eps_w)",
                                      "_, _, _, u = layer_update_score([s.weight for s in g], [s.shadow for s in g], self.dtype, self.eps_w)"),
    "eps_in_numerator_too": ("np.float64(A / n) / np.float64(B / n + eps_w)", "np.float64(A / n + eps_w) / np.float64(B / n + eps_w)"),
    "restore_strict_t_fail": ('if v["step"] <= t_fail and v["mask"][l]:', 'if v["step"] < t_fail and v["mask"][l]:'),
    "select_resets_every_timestamp": ("            if mask[l]:  # Eq. 4: reset on persist\n                self.delta[l] = 0.0\n                self.t_last[l] = step",
                                      "            if mask[l]:  # Eq. 4: reset on persist\n                self.delta[l] = 0.0\n            self.t_last[l] = step"),
    "weighted_age_over_layer_count": ('            "weighted_age": float(num) / float(den),', '            "weighted_age": float(num) / float(self.N),'),
    "stats_max_age_is_min": ('            "max_age": max(ages),', '            "max_age": min(ages),'),
    "pack_reports_done_early": ('"next_rank": last, "done": int(last == len(sel))}', '"next_rank": last, "done": 1}'),
    "weighted_by_count_not_size": ("num = sum(self.n[l] * ages[l] for l in range(self.N))",
                                   "num = sum(ages[l] for l in range(self.N)) * sum(self.n) // self.N"),
    "rebase_keeps_delta": ("            self.delta[l] = 0.0\n            self.t_last[l] = step\n            for s in g:",
                           "            self.t_last[l] = step\n            for s in g:"),
    "rebase_keeps_timestamps": ("            self.delta[l] = 0.0\n            self.t_last[l] = step\n            for s in g:",
                                "            self.delta[l] = 0.0\n            for s in g:"),
    "rebase_keeps_shadow": ("                if s.shadow is not None:\n                    s.shadow[...] = s.weight",
                            "                pass"),
    "capacity_off_by_record": ("total + self.R[sel[last]] <= capacity", "total + self.R[sel[last]] < capacity"),
    "adamw_no_bias_correction": ('"c1": f(1.0 / (1.0 - beta1 ** t)), "c2": f(1.0 / (1.0 - beta2 ** t)),',
                                 '"c1": f(1.0), "c2": f(1.0),'),
    "adamw_coupled_decay": ("    g = g.astype(f)\n    m_new", "    g = (g.astype(f) + (1.0 - sc['decay']) / sc['lr'] * p).astype(f) if decayed else g.astype(f)\n    m_new"),
    "adamw_decay_ignores_group": ("p1 = (p * sc[\"decay\"]).astype(f) if decayed else p.astype(f)\n    p_new =",
                                  "p1 = (p * sc[\"decay\"]).astype(f)\n    p_new ="),
    "sgd_decay_ignores_group": ("p1 = (p * sc[\"decay\"]).astype(f) if decayed else p.astype(f)\n    return (p1 -",
                                "p1 = (p * sc[\"decay\"]).astype(f)\n    return (p1 -"),
    "sgd_sign_flipped": ("return (p1 - (sc[\"lr\"] * g.astype(f)).astype(f)).astype(f)",
                         "return (p1 + (sc[\"lr\"] * g.astype(f)).astype(f)).astype(f)"),
    "sgd_decay_without_lr": ("return {\"lr\": f(lr), \"decay\": f(1.0 - lr * weight_decay)}",
                          "return {\"lr\": f(lr), \"decay\": f(1.0 - weight_decay)}"),
    "adamw_eps_inside_sqrt": ("denom = (np.sqrt(v_hat).astype(f) + sc[\"eps\"]).astype(f)",
                              "denom = np.sqrt((v_hat + sc[\"eps\"]).astype(f)).astype(f)"),
    "adamw_drift_on_new_params": ("_, _, _, u = layer_update_score([s._p_new for s in g], [s._p_old for s in g], DT_F32, self.eps_w)",
                                  "_, _, _, u = layer_update_score([s._p_old for s in g], [s._p_new for s in g], DT_F32, self.eps_w)"),
    "adamw_weights_not_rounded": ("s.weight[...] = bf16_round(p_new) if self.dtype == DT_BF16 else p_new",
                                  "s.weight[...] = (p_new.view(np.uint32) >> 16).astype(np.uint16) if self.dtype == DT_BF16 else p_new"),
    "bf16_ties_away": ("r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)",
                       "r = ((b + np.uint64(0x8000)) >> np.uint64(16)).astype(np.uint16)"),
    "bf16_truncates": ("r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)",
                       "r = (b >> np.uint64(16)).astype(np.uint16)"),
    "bf16_ties_to_odd": ("r = ((b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)",
                         "r = ((b + np.uint64(0x8000) - ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)"),
    "bf16_nan_unquieted": ("        r[nan] = np.uint16(0x7FC0)", "        pass"),
    "resync_unpersist_keeps_reset": ("            self.delta[layer] = self._pre_delta[layer]\n", ""),
    "resync_unpersist_keeps_timestamp": ("            self.t_last[layer] = self._pre_t_last[layer]\n", ""),
    "resync_persist_keeps_delta": ("            self.mask[layer] = 1\n            self.delta[layer] = 0.0\n",
                                   "            self.mask[layer] = 1\n"),
    "resync_persist_no_timestamp": ("            self.t_last[layer] = self.mask_step\n", ""),
    "resync_persist_not_packed": ("            self.unpacked.add(layer)\n", ""),
    "resync_unpersist_still_packed": ("            self.unpacked.discard(layer)\n", ""),
    "accum_drops_unpacked_selection": ("if self.unpacked and (self.pending_persists or self.mode == MODE_SNAPSHOT):",
                                       "if self.unpacked and self.mode == MODE_SNAPSHOT:"),
    "rebase_selection_droppable": ("        self.unpacked = set(range(self.N))\n        self.pending_persists = True\n\n    def stats(",
                                   "        self.unpacked = set(range(self.N))\n\n    def stats("),
    "init_base_blocks_warmup": ("        self.pending_persists = False\n\n    def _require_packed",
                                "        self.pending_persists = True\n\n    def _require_packed"),
}


def mutant(name):
    old, new = MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation anchor for {name} not unique"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    sys.modules[mod.__name__] = mod
    exec(compile(SRC.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


def all_checks(M):
    yield lambda: [c(M.layer_update_score) for c in (
        P.check_closed_form, P.check_denominator_is_previous, P.check_joint_mean,
        P.check_zero_change, P.check_eps_in_denominator, P.check_scale_invariance,
        P.check_exact_rational)]
    cls = M.LayerCheckOracle
    yield lambda: P.check_bf16_round(M.bf16_round)
    for c in (P.check_ge_threshold, P.check_delta_in_fp64, P.check_k0_extremes, P.check_record_format,
              P.check_capacity,
              P.check_restore_errors, P.check_accum_equals_snapshot_first_step, P.check_resync,
              P.check_call_order_errors, P.check_record_format_weights_only, P.check_fused_step_rules,
              P.check_snapshot_partial_pack_refresh, P.check_layout_validation,
              P.check_unpacked_selection_blocks):
        yield lambda c=c: c(cls)
    for mode in (O.MODE_ACCUM, O.MODE_SNAPSHOT):
        yield lambda mode=mode: P.check_staleness_period(cls, mode)
        yield lambda mode=mode: P.check_irregular_steps(cls, mode)
        yield lambda mode=mode: P.check_stats_invariants(cls, mode)
        yield lambda mode=mode: P.check_restore_roundtrip(cls, mode)
        yield lambda mode=mode: P.check_rebase(cls, mode)
    yield lambda: M.record_bytes([128], 2, True) == 14 * 128 or (_ for _ in ()).throw(AssertionError())
    for mode in (O.MODE_ACCUM, O.MODE_SNAPSHOT):
        yield lambda mode=mode: run_bruteforce(M, mode, O.DT_BF16, 0, steps=12)
    for chk in (A.test_first_step_is_lr_times_sign, A.test_decoupled_weight_decay_on_zero_gradient,
                A.test_matches_torch_adamw_over_steps, A.test_eps_beside_the_root, A.test_fused_step_drift_is_eq1_on_the_parameters,
                G.test_closed_form_exact, G.test_decay_and_gradient_together, G.test_decoupled_weight_decay,
                G.test_matches_torch_sgd,
                G.test_drift_is_eq1_on_the_parameters):
        yield lambda chk=chk: chk(M)


def test_unmutated_passes_everything():
    mod = types.ModuleType("oracle_copy")
    sys.modules[mod.__name__] = mod
    exec(compile(SRC, "<copy>", "exec"), mod.__dict__)
    for chk in all_checks(mod):
        chk()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    M = mutant(name)
    for chk in all_checks(M):
        try:
            chk()
        except Exception:
            return
    pytest.fail(f"planted mistake {name!r} passed every pin")
