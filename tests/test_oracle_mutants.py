"""The pins catch plausible mistakes.  Each case plants one mistake in a copy
of the oracle's source (never in the oracle itself), compiles it, points the
oracle module at the mutant, and requires the matching pin test to fail."""
import ctypes as C
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "frog_oracle.c")

# (name, text in frog_oracle.c, replacement, pin tests that must fail)
MUTANTS = [
    ("distance sign", "double t = (double)a[i] - (double)b[i];", "double t = (double)a[i] + (double)b[i];",
     ["test_dist_matches_numpy_fp64"]),
    ("distance drops a term", "for (int i = 0; i < d; ++i) {\n        double t = (double)a[i]",
     "for (int i = 1; i < d; ++i) {\n        double t = (double)a[i]", ["test_dist_exact_small_integers"]),
    ("lower bound uses <=", "if (attr_sorted[mid] < lo) a = mid + 1;", "if (attr_sorted[mid] <= lo) a = mid + 1;",
     ["test_rank_bounds_match_searchsorted"]),
    ("hotspot boundary term", "int64_t bl = el + 1, br = sr;", "int64_t bl = el, br = sr;",
     ["test_hotspot_hand_examples", "test_hotspot_bruteforce"]),
    ("hotspot descent bound", "while (d < H - 1) {\n        int64_t mid = L + (R - L) / 2;\n        if (r <= mid) R = mid;",
     "while (d < H) {\n        int64_t mid = L + (R - L) / 2;\n        if (r <= mid) R = mid;",
     ["test_hotspot_hand_examples", "test_hotspot_bruteforce"]),
    ("range test off by one", "if (v != FO_NONE && v >= l && v <= r) {", "if (v != FO_NONE && v >= l && v < r) {",
     ["test_en_ident_hand_examples"]),
    ("budget stops one early", "if (cnt == B) return cnt;", "if (cnt + 1 >= B) return cnt;",
     ["test_en_ident_hand_examples"]),
    ("stratum bound", "int64_t s = l + (j * cnt) / epn;", "int64_t s = l + (j * cnt) / (epn + 1);",
     ["test_entry_points_stratified_distinct_in_range"]),
    ("shared threshold rounds down", "uint64_t t = (((uint64_t)E << 32) + (uint64_t)cnt - 1) / (uint64_t)cnt;",
     "uint64_t t = ((uint64_t)E << 32) / (uint64_t)cnt;", ["test_entry_threshold_closed_form"]),
    ("shared sample keeps the threshold", "if ((uint64_t)fo_entry_priority(seed, i) < T) out[c++]",
     "if ((uint64_t)fo_entry_priority(seed, i) <= T + 20000000) out[c++]", ["test_entry_points_shared_membership"]),
    ("shared priority low word", "return (uint32_t)(fo_splitmix64(fo_splitmix64(seed) ^ (uint64_t)i) >> 32);",
     "return (uint32_t)fo_splitmix64(fo_splitmix64(seed) ^ (uint64_t)i);", ["test_entry_priority_is_splitmix_high_word"]),
    ("shared priority seed unmixed", "return (uint32_t)(fo_splitmix64(fo_splitmix64(seed) ^ (uint64_t)i) >> 32);",
     "return (uint32_t)(fo_splitmix64(seed ^ (uint64_t)i) >> 32);", ["test_entry_points_shared_size_nesting_and_sharing"]),
    ("eager check does not skip visited",
     "if (v != FO_NONE && v >= l && v <= r && fo_visited_insert(vis, v)) {",
     "if (v != FO_NONE && v >= l && v <= r && (fo_visited_insert(vis, v) || 1)) {",
     [("test_search_ablations_equal_textbook", dict(hot_mode=0, eager=True))]),
    ("hotspot ablation keeps one layer less", "if (hot_mode == 1) Le = ix->H - 1;", "if (hot_mode == 1) Le = ix->H - 2;",
     [("test_search_ablations_equal_textbook", dict(hot_mode=1, eager=False))]),
    ("tie order reversed", "if (a->id < b->id) return -1;\n    if (a->id > b->id) return 1;\n    return 0;\n}\n\n/* A visited",
     "if (a->id < b->id) return 1;\n    if (a->id > b->id) return -1;\n    return 0;\n}\n\n/* A visited",
     ["test_exact_breaks_distance_ties_by_rank"]),
    ("pool truncation", "np = np + nnew < L ? np + nnew : L;", "np = np + nnew < L ? np + nnew : L - 1;",
     ["test_search_full_range_equals_textbook_greedy"]),
    ("visited check skipped", "            if (eager || fo_visited_insert(vis, v)) {\n                work[np + nnew].dist = fo_dist(q,",
     "            if (eager || fo_visited_insert(vis, v) || 1) {\n                work[np + nnew].dist = fo_dist(q,",
     ["test_search_invariants_tiny_workload"]),
    ("fusion weight", "double w = 1.0 - beta * (1.0 - pow(da, gamma));", "double w = 1.0 - beta * pow(da, gamma);",
     ["test_fusion_special_values"]),
    ("fusion attribute scale", "double da = (double)diff / (double)(seglen - 1);",
     "double da = (double)diff / (double)seglen;", ["test_fusion_special_values"]),
    ("leaf keeps farthest", "qsort(fu, (size_t)c, sizeof(fo_ranked), fo_ranked_cmp);\n                    qsort(ve",
     "qsort(fu, (size_t)c, sizeof(fo_ranked), fo_ranked_cmp);\n                    for (int z = 0; z < c / 2; ++z) { fo_ranked tz = fu[z]; fu[z] = fu[c - 1 - z]; fu[c - 1 - z] = tz; }\n                    qsort(ve",
     ["test_build_leaf_layer_is_exact_fusion_topm"]),
    # construction's inductive step (Sec 6.1) and patience (Sec 6.2.2)
    ("rng comparison reversed", "if (dck < cand[i].dist) { ok = 0; break; }",
     "if (dck > cand[i].dist) { ok = 0; break; }", ["test_rng_prune_hand_1d", "test_rng_prune_hand_2d"]),
    ("rng prunes ties", "if (dck < cand[i].dist) { ok = 0; break; }",
     "if (dck <= cand[i].dist) { ok = 0; break; }", ["test_rng_prune_tie_keeps_candidate"]),
    ("rng tops up with the farthest", "for (int i = 0; i < nc && nk < m; ++i) {\n        if (!kept[i])",
     "for (int i = nc - 1; i >= 0 && nk < m; --i) {\n        if (!kept[i])", ["test_rng_prune_hand_1d"]),
    ("patience stops late", "if (left <= 0) break;", "if (left < 0) break;",
     [("test_sibling_search_patience_chain", dict(patience=4))]),
    ("patience stops early", "int left = patience;\n    int64_t nexp", "int left = patience - 1;\n    int64_t nexp",
     ["test_sibling_search_all_seeded_is_exact_topm"]),
    ("improved tested over the whole pool", "int top = nnp < m ? nnp : m;", "int top = nnp;",
     [("test_sibling_search_patience_chain", dict(patience=4))]),
    ("patience never reset", "if (improved) left = patience;", "if (improved) left = left + 0;",
     ["test_sibling_search_patience_resets_on_improvement"]),
    ("sibling is the own child", "if (u <= mid) { ts = mid + 1; te = e; } else { ts = s; te = mid; }",
     "if (u <= mid) { ts = s; te = mid; } else { ts = mid + 1; te = e; }", ["test_build_all_seeded_equals_restatement"]),
    ("child m-ANN dropped", "int32_t v = PG[u * m + t];\n                        if (v == FO_NONE) continue;",
     "int32_t v = PG[u * m + t];\n                        if (v == FO_NONE || 1) continue;",
     ["test_build_all_seeded_equals_restatement"]),
    ("fusion re-rank on the child length", "fus[t].key = fo_fusion(cand[t].dist, u, cand[t].id, len, beta, gamma);",
     "fus[t].key = fo_fusion(cand[t].dist, u, cand[t].id, len / 2 + 1, beta, gamma);",
     ["test_build_all_seeded_equals_restatement"]),
    ("parent graph keeps the unpruned list", "fo_rng_prune(X_rank, d, cand, nc, m, PGn + u * m);",
     "for (int t = 0; t < m; ++t) PGn[u * m + t] = t < nc ? cand[t].id : FO_NONE;",
     ["test_build_all_seeded_equals_restatement"]),
]


@pytest.mark.parametrize("name,old,new,tests", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, old, new, tests, tmp_path, monkeypatch):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site not found: {name}"
    mutated = src.replace(old, new, 1)
    c_path = tmp_path / "mutant.c"
    so_path = tmp_path / "libmutant.so"
    c_path.write_text(mutated)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                           "-w", "-o", str(so_path), str(c_path), "-lm"])
    mutant = oracle.configure(C.CDLL(str(so_path)))
    monkeypatch.setattr(oracle, "_lib", mutant)
    for tname in tests:
        kwargs = {}
        if isinstance(tname, tuple):
            tname, kwargs = tname[0], dict(tname[1])
        fn = getattr(pins, tname)
        if "tiny_index" in fn.__code__.co_varnames[:fn.__code__.co_argcount]:
            import workloads
            w = workloads.make("tiny", n=3000, nq=200)
            kwargs["tiny_index"] = (w, oracle.build(w.X, w.attr))
        argnames = fn.__code__.co_varnames[:fn.__code__.co_argcount]
        if "n" in argnames and "H" in argnames:
            kwargs.update(n=16, H=4)
        with pytest.raises(AssertionError):
            fn(**kwargs)
