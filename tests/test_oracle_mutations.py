"""Planted mistakes in the oracle must fail at least one pin.

Each case rewrites one expression of one oracle function (on the CPU, in
this process only), then runs the pins named for it and expects one of them
to fail.  This checks that the pins constrain every step of the oracle:
a dropped term, a wrong sign or index, or a transposed operand is caught.
"""
import inspect
import textwrap

import numpy as np
import pytest

from oracle import protokv_oracle as O
from tests import test_oracle_alloc as AL
from tests import test_oracle_ema as E
from tests import test_oracle_maintenance as M
from tests import test_oracle_pins as P
from tests import test_oracle_rope as R
from tests import test_oracle_warmup as WU

MUTATIONS = [
    # (function, original text, planted mistake, pins expected to catch it)
    ("minibatch_kmeans", "eta = F32(one / F32(count[k]))", "eta = F32(0.5)",
     [WU.test_single_centre_tracks_the_running_mean]),
    ("minibatch_kmeans", "c[k] = ((F32(one - eta) * c[k])", "c[k] = ((F32(one + eta) * c[k])",
     [WU.test_single_centre_tracks_the_running_mean]),
    ("learn_codebooks", "init = xg[np.arange(C) * (N // C)]", "init = xg[np.arange(C)]",
     [WU.test_learned_codebooks_recover_each_subspace_and_side]),
    ("learn_codebooks", "xg = res[:, g * Dp:(g + 1) * Dp]", "xg = res[:, g:g + Dp]",
     [WU.test_learned_codebooks_recover_each_subspace_and_side]),
    ("learn_codebooks", "for side, res in enumerate((res_k, res_v)):", "for side, res in enumerate((res_k, res_k)):",
     [WU.test_learned_codebooks_recover_each_subspace_and_side]),
    ("rope_rotate", "x1 * c - x2 * s", "x1 * c + x2 * s",
     [R.test_rotation_is_complex_multiplication_and_a_block_rotation_matrix]),
    ("rope_rotate", "(-2.0 * np.arange(h, dtype=np.float64) / D)", "(-1.0 * np.arange(h, dtype=np.float64) / D)",
     [R.test_rotation_is_complex_multiplication_and_a_block_rotation_matrix]),
    ("rope_rotate", "x1, x2 = x[..., :h], x[..., h:]", "x1, x2 = x[..., 0::2], x[..., 1::2]",
     [R.test_rotation_is_complex_multiplication_and_a_block_rotation_matrix]),
    ("fold_frame", "ka, kb = F32(one - al), F32(one - be)", "ka, kb = F32(one - al), F32(one - al)",
     [E.test_repeated_token_follows_the_geometric_closed_form]),
    ("fold_frame", "(al * kk).astype(F32)).astype(F32)", "(al * vv).astype(F32)).astype(F32)",
     [E.test_repeated_token_follows_the_geometric_closed_form]),
    ("fold_frame", "(kb * bank.sum_v[k]).astype(F32) + (be * vv)", "(kb * bank.sum_v[k]).astype(F32) + (al * vv)",
     [E.test_repeated_token_follows_the_geometric_closed_form]),
    ("fold_frame", "zk = pq_encode((kk - bank.sum_k[k])", "zk = pq_encode((kk - F32(0) * bank.sum_k[k])",
     [E.test_residual_is_taken_after_the_centre_update]),
    ("fold_frame", "zv = pq_encode((vv - bank.sum_v[k]).astype(F32)[None, :], codebooks[1])",
     "zv = pq_encode((vv - bank.sum_v[k]).astype(F32)[None, :], codebooks[0])",
     [E.test_residual_is_taken_after_the_centre_update]),
    ("synthesize", "c, pv = bank.sum_k[k].copy(), bank.sum_v[k].copy()",
     "c, pv = (bank.sum_k[k] / F32(bank.n[k])).astype(F32), bank.sum_v[k].copy()",
     [E.test_synthesis_uses_the_stored_centres]),
    ("assignment_costs", "cost = -cos +", "cost = cos +",
     [P.test_cost_matches_scipy_cosine_and_mahalanobis]),
    ("assignment_costs", "- 2.0 * Bxy[None, :]", "+ 2.0 * Bxy[None, :]",
     [P.test_cost_matches_scipy_cosine_and_mahalanobis]),
    ("assignment_costs", "(Cc[None, :] * dx * dx", "(A[None, :] * dx * dx",
     [P.test_cost_matches_scipy_cosine_and_mahalanobis]),
    ("assignment_costs", "> p.t_idle", ">= p.t_idle", [P.test_idle_term_counts_frames]),
    ("assignment_costs", "p.lambda_sp * d_mah", "p.lambda_sp * d_mah * d_mah",
     [P.test_cost_matches_scipy_cosine_and_mahalanobis]),
    ("assignment_costs", "d_mah = np.maximum(q, 0.0) if p.mah_squared", "d_mah = np.sqrt(np.maximum(q, 0.0)) if p.mah_squared",
     [P.test_squared_mahalanobis_cost_matches_scipy]),
    ("argmin_lowest", "idx = np.argmin(cost, axis=1)", "idx = np.argmax(cost, axis=1)",
     [P.test_zero_lambdas_is_spherical_kmeans_assignment]),
    ("spatial_coords", "F32(col + 0.5) / F32(grid_w)", "F32(row + 0.5) / F32(grid_w)",
     [P.test_coordinates_are_cell_centres]),
    ("pq_encode", "codes[:, g] = np.argmin(acc, axis=1)", "codes[:, g] = np.argmax(acc, axis=1)",
     [P.test_pq_encode_matches_cdist_argmin]),
    ("pq_encode", "sub = residuals[:, g * Dp:(g + 1) * Dp]", "sub = residuals[:, g:g + Dp]",
     [P.test_pq_encode_matches_cdist_argmin]),
    ("fold_frame", "bank.sum_k[k] = (bank.sum_k[k] + kk)", "bank.sum_k[k] = (bank.sum_k[k] + vv)",
     [P.test_means_equal_sum_over_mass_from_assignment_log]),
    ("fold_frame", "(bank.sq_v[k] + (vv * vv)", "(bank.sq_v[k] + (vv * kk)",
     [lambda: P.test_mass_moment_hist_conservation("fp32")]),
    ("fold_frame", "r_k = (keys[rest].astype(F32) - c_snap)", "r_k = (keys[rest].astype(F32) - p_snap)",
     [P.test_histograms_match_nearest_codeword_of_logged_residuals]),
    ("fold_frame", "codes_v = pq_encode(r_v, codebooks[1])", "codes_v = pq_encode(r_v, codebooks[0])",
     [P.test_histograms_match_nearest_codeword_of_logged_residuals]),
    ("fold_frame", "F32(eta * s[0]))", "F32(eta * s[1]))", [P.test_spatial_ema_closed_form]),
    ("fold_frame", "F32(eta * F32(ddx * ddy))", "F32(eta * F32(ddx * ddx))", [P.test_spatial_ema_closed_form]),
    ("fold_frame", "np.array([1.0, 0.0, 1.0], dtype=F32)", "np.array([1.0, 1.0, 1.0], dtype=F32)",
     [P.test_spatial_ema_closed_form]),
    ("fold_frame", "bank.tau[k] = pos[j]\n    return", "bank.tau[k] = t_frame\n    return",
     [P.test_means_equal_sum_over_mass_from_assignment_log]),
    ("fold_frame", "free = [k for k in range(p.capacity) if bank.n[k] == 0]",
     "free = [k for k in range(p.capacity) if bank.n[k] == 0][::-1]",
     [P.test_capacity_at_least_evicted_seeds_every_token]),
    ("decode_top_s", "(int(hist[g, c]) + 1)", "(int(hist[g, c]) + 2)",
     [lambda: P.test_beam_decode_is_exact_top_s(3, 5, 8, 3)]),
    ("decode_top_s", "expanded.sort(key=lambda e: _order_key(*e))",
     "expanded.sort(key=lambda e: (-e[0], e[1][::-1]))",
     [lambda: P.test_beam_decode_is_exact_top_s(3, 5, 8, 3)]),
    ("synthesize", "rv = [residual_from_codes(z, codebooks[1])", "rv = [residual_from_codes(z, codebooks[0])",
     [P.test_pseudo_tokens_from_brute_force_modes]),
    ("synthesize", "b = math.log(bank.n[k])", "b = math.log(bank.n[k] + 1)",
     [P.test_log_mass_bias_equals_duplicated_tokens]),
    ("attend", "/ math.sqrt(Q.shape[1])", "/ Q.shape[1]",
     [P.test_attend_matches_torch_sdpa_with_additive_mask]),
    ("maintain", "bank.sum_k[k] = (bank.sum_k[k] * r)", "bank.sum_k[k] = (bank.sum_k[k] * F32(1))",
     [M.test_aging_floors_the_mass_and_keeps_the_centre]),
    ("maintain", "(1.0 - p.gamma)", "(1.0 + p.gamma)", [M.test_aging_floors_the_mass_and_keeps_the_centre]),
    ("maintain", "> p.t_idle", ">= p.t_idle", [M.test_aging_floors_the_mass_and_keeps_the_centre]),
    ("maintain", "ci, cj = (bank.sum_k[i] / ni)", "ci, cj = (bank.sum_k[i] / F32(1))",
     [lambda: M.test_merge_uses_the_centre_updated_by_earlier_merges(0.3, 1)]),
    ("maintain", "if not dk < ek2", "if not dk <= ek2",
     [M.test_merge_thresholds_are_strict_and_need_both_centres]),
    ("maintain", "if not dv < ev2", "if False",
     [M.test_merge_thresholds_are_strict_and_need_both_centres]),
    ("maintain", "F32(ni * bank.mu[i, a])", "F32(nj * bank.mu[i, a])",
     [M.test_merge_adds_statistics_and_weights_the_spatial_mean]),
    ("maintain", "bank.sq_v[i] = (bank.sq_v[i] + bank.sq_v[j])", "bank.sq_v[i] = (bank.sq_v[i] + bank.sum_v[j])",
     [M.test_merge_adds_statistics_and_weights_the_spatial_mean]),
    ("maintain", "bank.hist_v[i] += bank.hist_v[j]", "bank.hist_v[i] += bank.hist_k[j]",
     [M.test_merge_adds_statistics_and_weights_the_spatial_mean]),
    ("maintain", "reversed(list(near))", "list(near)",
     [M.test_recycling_takes_near_tokens_newest_frame_first_in_raster_order]),
    ("maintain", "bank.n[j] = 0", "bank.n[j] = bank.n[j]",
     [M.test_merge_adds_statistics_and_weights_the_spatial_mean]),
    ("residual_variance", "total = total + np.maximum(e2 - m2, 0.0)", "total = total + np.maximum(e2, 0.0)",
     [AL.test_residual_variance_is_numpys_weighted_variance_of_the_codewords]),
    ("residual_variance", "mean = mean + pc[:, None] * cw[c][None, :]", "mean = mean + pc[:, None] * cw[0][None, :]",
     [AL.test_residual_variance_is_numpys_weighted_variance_of_the_codewords]),
    ("residual_variance", "for side, hist in ((0, bank.hist_k), (1, bank.hist_v)):",
     "for side, hist in ((0, bank.hist_k), (1, bank.hist_k)):",
     [AL.test_residual_variance_is_numpys_weighted_variance_of_the_codewords]),
    ("allocate_pseudo", "x.append(1.0 + rest * float(var[k]) / w)", "x.append(rest * float(var[k]) / w)",
     [lambda: AL.test_allocation_keeps_the_total_and_follows_the_exact_shares(2, 8, 16)]),
    ("allocate_pseudo", "cur = math.floor(X + 0.5)", "cur = math.floor(X)",
     [AL.test_allocation_special_cases]),
    ("allocate_pseudo", "over = [k for k in range(A) if not capped[k] and x[k] > s_max]",
     "over = [k for k in range(A) if not capped[k] and x[k] > s_max + 4]",
     [AL.test_allocation_special_cases]),
    ("synthesize", "Sk = int(counts[k])", "Sk = p.S",
     [AL.test_synthesis_gives_each_prototype_its_top_sk_modes]),
    ("_dist2", "for d in range(len(a64)):", "for d in range(len(a64) - 1):",
     [M.test_merge_distance_is_the_squared_euclidean_distance]),
    ("_dist2", "diff = a64[d] - b64[d]", "diff = a64[d] - b64[d - 1]",
     [M.test_merge_distance_is_the_squared_euclidean_distance]),
    ("_near_threshold", "return abs(d2 - eps2) <= NEAR_THRESHOLD_REL * eps2", "return False",
     [M.test_pair_on_the_threshold_is_counted_and_not_merged]),
    ("argmin_lowest", "margin = part[:, 1] - part[:, 0]", "margin = 0 * (part[:, 1] - part[:, 0])",
     [P.test_margin_is_second_best_minus_best_of_an_independent_cost_matrix]),
    ("argmin_lowest", "margin = part[:, 1] - part[:, 0]", "margin = 10 * (part[:, 1] - part[:, 0])",
     [P.test_margin_is_second_best_minus_best_of_an_independent_cost_matrix]),
    ("argmin_lowest", "margin = part[:, 1] - part[:, 0]", "margin = part[:, 2] - part[:, 0]",
     [P.test_margin_is_second_best_minus_best_of_an_independent_cost_matrix]),
    ("round_kv", "top = ((bits + 0x7FFF + lsb) >> 16)", "top = ((bits + 0 * lsb) >> 16)",
     [P.test_round_kv_bf16_is_torch_round_to_nearest_even]),
    ("round_kv", "top = ((bits + 0x7FFF + lsb) >> 16)", "top = ((bits + 0x8000 + 0 * lsb) >> 16)",
     [P.test_round_kv_bf16_is_torch_round_to_nearest_even]),
]


def _mutated(fn_name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(O, fn_name)))
    assert src.count(old) == 1, (fn_name, old)
    ns = dict(O.__dict__)
    exec(compile(src.replace(old, new), f"<mutant {fn_name}>", "exec"), ns)
    return ns[fn_name]


@pytest.mark.parametrize("case", range(len(MUTATIONS)))
def test_planted_mistake_is_caught(case, monkeypatch):
    fn_name, old, new, pins = MUTATIONS[case]
    monkeypatch.setattr(O, fn_name, _mutated(fn_name, old, new))
    caught = False
    for pin in pins:
        try:
            pin()
        except Exception:          # AssertionError or a crash both count
            caught = True
            break
    assert caught, f"mutation in {fn_name} ({new!r}) passed every pin"


def test_stream_eviction_mutation_is_caught(monkeypatch):
    """Evicting when the ring holds W frames (instead of more than W)."""
    src = textwrap.dedent(inspect.getsource(O.OracleStream))
    old = "if len(self.rings[0]) > self.p.window_frames:"
    assert src.count(old) == 1
    ns = dict(O.__dict__)
    exec(compile(src.replace(old, old.replace(">", ">=")), "<mutant stream>", "exec"), ns)
    monkeypatch.setattr(O, "OracleStream", ns["OracleStream"])
    with pytest.raises(Exception):
        P.test_capacity_limit_reproduces_exact_attention(1)


STREAM_MUTATIONS = [
    # (original text in OracleStream, planted mistake, pin expected to catch it)
    ("dataclasses.replace(self.p, use_pq=False)", "self.p",
     WU.test_warmup_folds_count_no_codes_and_fill_the_reservoir),
    ("rk[:room]]", "rk[:room][::-1]]", WU.test_reservoir_residuals_use_the_pre_fold_centres),
    ("P + np.repeat(np.arange(Tq), grp)", "np.repeat(np.arange(Tq), grp)",
     lambda: R.test_capacity_limit_with_rope_is_exact_positional_attention(1)),
    ("self.banks[u].tau[pseudo.slots]", "self.banks[u].n[pseudo.slots]",
     lambda: R.test_capacity_limit_with_rope_is_exact_positional_attention(8)),
    ("f * T + j for f in fr", "f * T for f in fr",
     lambda: R.test_capacity_limit_with_rope_is_exact_positional_attention(1)),
]


@pytest.mark.parametrize("case", range(len(STREAM_MUTATIONS)))
def test_stream_readout_mutation_is_caught(case, monkeypatch):
    """Planted mistakes in the stream's rotary positions (query, pseudo-token
    anchor, near tokens)."""
    old, new, pin = STREAM_MUTATIONS[case]
    src = textwrap.dedent(inspect.getsource(O.OracleStream))
    assert src.count(old) == 1, old
    ns = dict(O.__dict__)
    exec(compile(src.replace(old, new), "<mutant stream>", "exec"), ns)
    monkeypatch.setattr(O, "OracleStream", ns["OracleStream"])
    with pytest.raises(Exception):
        pin()
