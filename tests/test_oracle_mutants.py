"""Plant a plausible mistake in a copy of the oracle (on the CPU) and check
that at least one pin fails.  This is evidence that the pins constrain every
step: the group max, the window edge, the local mass, the bias, the scale, the
routing query, tie-breaking, the backward's chunk and score terms, and the
landmark compression's entropy, head-to-group map and both backward terms, and
the per-head normalisation of the selection variant."""
import os

import pytest

import oracle
from tests import test_oracle_headnorm as hnorm
from tests import test_oracle_landmark as lmk
from tests import test_oracle_pins as pins

SRC = open(oracle._SRC).read()

MUTANTS = {
    "group_score_first_head_only": ("if (sh[c] - lse > sigma[c]) sigma[c] = sh[c] - lse;",
                                    "if (hh == 0) sigma[c] = sh[c] - lse;",
                                    [pins.test_hand_worked_example]),
    "window_edge_off_by_one": ("long lc = floor_div(i - W + 1, S);", "long lc = floor_div(i - W, S);",
                               [pins.test_hand_worked_example]),
    "local_mass_misweighted": ("logits[0] = lam0;\n            for (int r = 0; r < st->nsel; ++r) logits[1 + r] = st->shat[r];",
                               "logits[0] = lam0 - 1.0;\n            for (int r = 0; r < st->nsel; ++r) logits[1 + r] = st->shat[r];",
                               [lambda: pins.test_p1_chunk1_window1_topall_is_dense_causal(4, 1, 4)]),
    "bias_dropped": ("+ BIAS(in, b, hl, c);", ";",
                     [lambda: pins.test_p2_exact_mass_landmarks_top_all_is_dense_causal(4, 5, 50, 2, 1, 2)]),
    "scale_missing_in_surrogate": ("return (REAL)p->scale * dot_f(QHAT", "return dot_f(QHAT",
                                   [lambda: pins.test_p1_chunk1_window1_topall_is_dense_causal(1, 1, 1)]),
    "routing_query_ignored": ("const float* base = in->q_route ? in->q_route : in->q;", "const float* base = in->q;",
                              [lambda: pins.test_p7_backward_matches_finite_differences(True, True, True)]),
    "ties_to_larger_index": ("sigma[c] > sigma[best]) best = c;", "sigma[c] >= sigma[best]) best = c;",
                             [pins.test_ties_go_to_the_smaller_chunk_index]),
    "bwd_chunk_uses_global_u": ("REAL ds = a * pj * (gv - uc);", "REAL ds = a * pj * (gv - ubar);",
                                [lambda: pins.test_p7_backward_matches_finite_differences(True, True, True)]),
    "bwd_score_grad_drops_u": ("REAL dshat = a * (uc - ubar);", "REAL dshat = a * uc;",
                               [lambda: pins.test_p7_backward_matches_finite_differences(False, False, True)]),
    # per-head normalised selection (Sec. 4.1 variant)
    "head_norm_skipped": ("const REAL lse = p->head_norm && ncand > 0 ? logsumexp(sh, ncand) : 0;",
                          "const REAL lse = 0;",
                          [hnorm.test_hand_worked_example,
                           hnorm.test_a_shift_of_one_heads_scores_changes_only_the_raw_selection]),
    # landmark compression (Prop. 3.1)
    "lmk_entropy_sign": ("ent -= pj * logp;", "ent += pj * logp;", [lmk.test_entropy_range_and_uniform_regime]),
    "lmk_group_map": ("return hl / (p->Hl / p->Hkv);", "return hl % p->Hkv;",
                      [lambda: lmk.test_taylor_point_identity_and_gradient(True)]),
    "lmk_bwd_drops_entropy_term": ("gp[j] = dot_f(dkc, kj, d) - db * (logp + 1);", "gp[j] = dot_f(dkc, kj, d);",
                                   [lmk.test_taylor_identity_gives_a_null_direction]),
    "lmk_bwd_drops_key_summary_term": ("dkj[u] += pr[j] * (REAL)dkc[u] + p->scale * ds * (REAL)qc[u];",
                                       "dkj[u] += p->scale * ds * (REAL)qc[u];",
                                       [lambda: lmk.test_backward_matches_finite_differences(True, False)]),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new, checks = MUTANTS[name]
    assert SRC.count(old) == 1, f"mutation anchor for {name} not unique"
    lib = oracle.build_variant(SRC.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    with oracle.swapped_library(lib):
        for check in checks:
            with pytest.raises(AssertionError):
                check()
