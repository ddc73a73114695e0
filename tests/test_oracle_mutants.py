"""Planted mistakes: each case compiles a copy of the oracle's C source with
one plausible error and checks that the pins named for it fail.  This shows
the pins constrain the oracle, not only that the oracle agrees with itself.
CPU only; each case is a gcc build plus one pytest subprocess."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "ssref.c")

# (name, text in ssref.c, replacement, pins expected to catch it)
MUTANTS = [
    ("draw_takes_ge", "    if (cum > target) { pick = r; break; }", "    if (cum >= target) { pick = r; break; }",
     "test_draw_golden"),
    ("min_p_threshold_shifted", "int keep = l >= lt, near = m < SSREF_NEAR;",
     "int keep = l >= lt + 0.05, near = m < SSREF_NEAR;", "test_min_p_keeps_tokens"),
    ("top_p_unnormalised", "    double thr = (double)top_p * Zk;", "    double thr = (double)top_p;",
     "test_top_p_is_minimal_prefix"),
    ("repetition_penalty_flipped", "v = (v > 0.0f) ? v / rep : v * rep;", "v = (v > 0.0f) ? v * rep : v / rep;",
     "test_prologue_golden"),
    ("frequency_term_dropped", "float t = freq * (float)c[i]; v = v - t;", "float t = freq * (float)c[i]; (void)t;",
     "test_prologue_golden"),
    ("philox_key_schedule", "    k0 += 0x9E3779B9u;", "    k0 += 0x9E3779B7u;", "test_philox_published_vectors"),
    ("ties_take_higher_index", "  return (p->i < q->i) ? -1 : (p->i > q->i);", "  return (p->i > q->i) ? -1 : (p->i < q->i);",
     "test_topk_matches_lexsort or test_greedy_ties_take_lowest_index"),
    # near-boundary band (admissible outcomes) and the Philox counter layout
    ("top_p_band_always_open", "int keep = excl < thr, near = m < SSREF_NEAR;", "int keep = excl < thr, near = 1;",
     "test_top_p_boundary_distance or test_sample_admits_both"),
    ("min_p_band_too_wide", "int keep = l >= lt, near = m < SSREF_NEAR;", "int keep = l >= lt, near = m < 1e-2;",
     "test_min_p_boundary_distance"),
    ("draw_band_closed", "    int before = prev <= target || fabs(prev - target) < band;",
     "    int before = prev <= target;", "test_draw_boundary_distance"),
    ("draw_margin_always_zero", "    *margin = (Z > 0.0) ? m / Z : 0.0;", "    *margin = 0.0;",
     "test_draw_boundary_distance"),
    ("acceptance_band_closed", "        near = m < SSREF_NEAR;", "        near = 0;",
     "test_verify_admits_accept_and_reject"),
    ("logprob_normaliser_over_listed_tokens", "      for (int r = 0; r < nv; ++r) Z += exp(((double)y[order[r]] - M) / tau);",
     "      for (int r = 0; r < (n_lp < nv ? n_lp : nv); ++r) Z += exp(((double)y[order[r]] - M) / tau);",
     "test_logprobs_match_scipy_log_softmax"),
    ("logprob_temperature_ignored",
     "      if ((em & R_TEMP) && !(em & R_GREEDY) && p->temperature[b] > 0.0f) tau = (double)p->temperature[b];",
     "      if ((em & R_TEMP) && !(em & R_GREEDY) && p->temperature[b] > 0.0f) tau = 1.0;",
     "test_logprobs_temperature_scales_differences"),
    ("sparse_q_last_entry_wins", "    if (c->qi[o + i] == id) s += (double)c->qv[o + i];",
     "    if (c->qi[o + i] == id) s = (double)c->qv[o + i];", "test_verify_sparse_first_token"),
    ("sparse_q_first_position_list", "  const int64_t o = ((int64_t)c->b * c->L + (l - 1)) * c->kq;",
     "  const int64_t o = ((int64_t)c->b * c->L) * c->kq;", "test_verify_sparse_lists_are_per_position"),
    ("gumbel_noise_added", "    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) - (double)g[order[r]];",
     "    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) + (double)g[order[r]];", "test_gumbel_draw"),
    ("gumbel_temperature_dropped", "    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) - (double)g[order[r]];",
     "    double sc = ((yr == M) ? 0.0 : (yr - M)) - (double)g[order[r]];", "test_gumbel_draw"),
    ("gumbel_noise_by_rank", "    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) - (double)g[order[r]];",
     "    double sc = ((yr == M) ? 0.0 : (yr - M) / tau) - (double)g[r];", "test_gumbel_draw"),
    ("tree_map_ignored", "    if (t >= 0 && t < c->Lt) src = (int64_t)c->b * c->Lt + t;",
     "    if (t >= 0 && t < c->Lt) src = (int64_t)c->b * c->Lt + (l - 1);", "test_verify_tree_rows_are_selected"),
    ("tree_request_stride_of_the_path", "    if (t >= 0 && t < c->Lt) src = (int64_t)c->b * c->Lt + t;",
     "    if (t >= 0 && t < c->Lt) src = (int64_t)c->b * (c->L + 1) + t;", "test_verify_tree_rows_are_selected"),
    ("full_row_uses_bounded_normaliser", "    if (full) row_distribution(y, order, nv, mode, tmp, tk, tp, mp, nv, wf, &df);",
     "    if (full) row_distribution(y, order, nv, mode, tmp, tk, tp, mp, cap, wf, &df);",
     "test_full_row_top_p_uses_the_whole_row"),
    ("full_row_fit_test_inclusive", "static int full_fits(int ns, int k_cap) { return ns < k_cap; }",
     "static int full_fits(int ns, int k_cap) { return ns <= k_cap; }",
     "test_full_row_overflow_falls_back"),
    ("uniform_counter_words_swapped", "  uint32_t ctr[4] = {request, (uint32_t)((uint64_t)position & 0xFFFFFFFFu),",
     "  uint32_t ctr[4] = {(uint32_t)((uint64_t)position & 0xFFFFFFFFu), request,",
     "test_uniform_counter_words"),
]


@pytest.mark.parametrize("name,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new, pins):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    mut = tmp_path / "ssref_mut.c"
    mut.write_text(src.replace(old, new))
    so = tmp_path / "libssref_mut.so"
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-shared", "-fPIC", "-o", str(so),
                    str(mut), "-lm"], check=True)
    env = dict(os.environ, SSREF_LIB=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"), "-k", pins],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert "failed" in r.stdout or "passed" in r.stdout, r.stdout[-2000:]  # the selected pins ran
    assert r.returncode == 1, f"{name}: the pins ({pins}) did not catch the planted mistake\n{r.stdout[-2000:]}"
