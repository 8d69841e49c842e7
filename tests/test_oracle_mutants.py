"""Mutation check of the pins: each plausible mistake planted in a copy of
oracle.c (built on the CPU into a temporary library) must fail at least one
of the oracle's pin tests.  The real oracle is never modified."""
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle

import test_oracle_bruteforce as t_bf
import test_oracle_independent as t_ind
import test_oracle_paper_examples as t_pap
import test_oracle_properties as t_prop
import test_oracle_search as t_search
import test_oracle_phi as t_phi
import test_oracle_victim as t_vic
import test_oracle_batch as t_batch
import test_oracle_prefix as t_prefix
import test_oracle_replica as t_rep
import test_oracle_search_rules as t_rules

# (name, original fragment, planted mistake)
MUTANTS = [
    # replica cap
    ("replica cap inclusive", "if (copies > w->replica_cap[m]) return 1;", "if (copies >= w->replica_cap[m]) return 1;"),
    ("replica cap counts only loads", "(((held[d] | loaded[d]) >> m) & 1u)", "((loaded[d] >> m) & 1u)"),
    ("replica cap counts only holders", "(((held[d] | loaded[d]) >> m) & 1u)", "((held[d] >> m) & 1u)"),
    ("replica cap skips the last level",
     "if (n_units > 0 && replica_over(w, res_level, loaded_level)) sc.status |= ORC_REPLICA;", ""),
    ("replica loads accumulate across levels", "          loaded_level[e] = 0;\n", ""),
    ("replica flag clears other bits", "sc.status |= ORC_REPLICA;\n        for", "sc.status = ORC_REPLICA;\n        for"),
    # rule-guided candidates (BestFeasibleBinding, PlanPrefetch)
    ("rules: residency ignored", "if (l < 0 || !((w->init_resident[d] >> m) & 1u)) continue;", "if (l < 0 || 1) continue;"),
    ("rules: slowest resident replica", "if (!resident || l < w->lat_us[(int64_t)i * D + b]) b = d;",
     "if (!resident || l > w->lat_us[(int64_t)i * D + b]) b = d;"),
    ("rules: value ratio inverted", "const __int128 x = (__int128)ud * lb, y = (__int128)ub * ld;",
     "const __int128 x = (__int128)ud * ld, y = (__int128)ub * lb;"),
    ("rules: free load not preferred", "if ((ld == 0) != (lb == 0)) cmp = ld == 0 ? 1 : -1;",
     "if ((ld == 0) != (lb == 0)) cmp = ld == 0 ? -1 : 1;"),
    ("rules: equal values keep the first", "if (cmp > 0 || (cmp == 0 && l < w->lat_us[(int64_t)i * D + b])) b = d;",
     "if (cmp > 0) b = d;"),
    ("rules: unlock counts waiting work", "    if (!ready[i]) continue;\n    for (int32_t d = 0; d < D; ++d) {",
     "    for (int32_t d = 0; d < D; ++d) {"),
    ("rules: readiness ignores arrival", "w->pred_off[i] == w->pred_off[i + 1] && w->wf_arrival_us[w->act_wf[i]] <= 0;",
     "w->pred_off[i] == w->pred_off[i + 1];"),
    ("rules: release ignores run times", "if (rel_lb[p] + (fast < 0 ? 0 : fast) > r) r = rel_lb[p] + (fast < 0 ? 0 : fast);",
     "if (rel_lb[p] > r) r = rel_lb[p];"),
    ("rules: release from the slowest device", "if (l >= 0 && (fast < 0 || l < fast)) fast = l;",
     "if (l >= 0 && (fast < 0 || l > fast)) fast = l;"),
    ("rules: prefetch without slack", "rel_lb[i] <= ld + w->prefetch_slack_us;", "rel_lb[i] <= ld;"),
    ("rules: prefetch of ready work", "const int on = !ready[i] && rel_lb[i]", "const int on = rel_lb[i]"),
    ("rules: prefetch on the incumbent's device", "const int32_t d = cd[i];\n        if (d < 0 || d >= D) continue;",
     "const int32_t d = dev[i];\n        if (d < 0 || d >= D) continue;"),
    ("rules: prefetch toggles", "cf[i / 4] = on ? (uint8_t)(cf[i / 4] | bit) : (uint8_t)(cf[i / 4] & ~bit);",
     "cf[i / 4] ^= bit;"),
    ("rules: binding falls back to uniform", "if (kind == 0 && mode == ORC_SEARCH_RULES) {", "if (kind == 0 && mode == 99) {"),
    # candidate generator
    ("philox multiplier swapped", "(uint64_t)0xD2511F53u * x0", "(uint64_t)0xCD9E8D57u * x0"),
    ("philox key not bumped", "k1 += 0xBB67AE85u;", ""),
    ("mutation kind from the low bits", "r[0] >> 30", "r[0] & 3u"),
    ("mutation site from the wrong word", "scale32(r[1], (uint32_t)N)", "scale32(r[2], (uint32_t)N)"),
    ("swap partner outside the level", "const int32_t j = lo + (int32_t)scale32(r[2], (uint32_t)(hi - lo));",
     "const int32_t j = (int32_t)scale32(r[2], (uint32_t)N);"),
    ("re-place ignores eligibility", "          if (w->lat_us[(int64_t)i * D + d] < 0) continue;\n          if (pick == 0) {",
     "          if (pick == 0) {"),
    ("fuse flip toggles prefetch", "cf[i / 4] ^= (uint8_t)(1u << (2 * (i % 4)));", "cf[i / 4] ^= (uint8_t)(1u << (2 * (i % 4) + 1));"),
    ("counter words swapped", "{(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)t, 0u}",
     "{(uint32_t)t, (uint32_t)(c >> 32), (uint32_t)c, 0u}"),
    ("release ignores arrival", "int64_t r = w->wf_arrival_us[wf];", "int64_t r = 0;"),
    ("victim prefers live copies", "if (alive2 < aliveV) victim = m2;", "if (alive2 > aliveV) victim = m2;"),
    ("victim most recently used", "} else if (last[d * M + m2] < last[d * M + victim]) {",
     "} else if (last[d * M + m2] > last[d * M + victim]) {"),
    ("prefetch ignored",
     "int64_t t = max64(max64(miss && pf[h] ? w->wf_arrival_us[wf] : r, free_before), dispatched[d]);",
     "int64_t t = max64(max64(r, free_before), dispatched[d]);"),
    ("peak without activation memory",
     "if (used[d] + run_act + Mx > peak[d]) peak[d] = used[d] + run_act + Mx;",
     "if (used[d] + run_act > peak[d]) peak[d] = used[d] + run_act;"),
    ("start ignores release after load", "s = max64(r, le);", "s = le;"),
    ("p95 rank rounded", "(95 * W + 99) / 100", "(95 * W + 50) / 100"),
    ("priority ignored", "if (x->prio != y->prio) return x->prio < y->prio ? -1 : 1;", ""),
    ("level ignored", "if (x->level != y->level) return x->level < y->level ? -1 : 1;", ""),
    ("fusion ignores deployment", " && w->act_model[u] == w->act_model[v]", ""),
    ("fusion ignores fan-out", "s->fusible[v] = (s->n_succ[u] == 1 &&", "s->fusible[v] = (s->n_succ[u] >= 1 &&"),
    ("member runs on its own device", "finish[v] = s + w->lat_us[(int64_t)v * D + d];",
     "finish[v] = s + w->lat_us[(int64_t)v * D + (pdev[v] >= 0 && pdev[v] < D ? pdev[v] : d)];"),
    ("makespan from time zero", "sc.makespan_us = max_fin - min_arr;", "sc.makespan_us = max_fin;"),
    ("load table transposed", "w->load_us[m * D + d]", "w->load_us[(d * M + m) % (M * D)]"),
    ("capacity check inclusive", "const int fits = !(used[d] + run_act + need > w->dev_cap_mib[d]);",
     "const int fits = !(used[d] + run_act + need >= w->dev_cap_mib[d]);"),
    ("eviction ignores activation memory",
     "int64_t need = (miss ? (int64_t)w->model_mib[m] : 0) + Mx;",
     "int64_t need = (miss ? (int64_t)w->model_mib[m] : 0);"),
    ("objective weight swapped", "float y = w->w_p95 * b;", "float y = w->w_makespan * b;"),
    ("hit ignores busy device",
     "int64_t t = max64(max64(miss && pf[h] ? w->wf_arrival_us[wf] : r, free_before), dispatched[d]);",
     "int64_t t = miss ? max64(max64(pf[h] ? w->wf_arrival_us[wf] : r, free_before), dispatched[d]) : r;"),
    ("loads double counted", "n_loads += 1;", "n_loads += 2;"),
    ("evicts one too many", "while (used[d] + run_act + need > w->dev_cap_mib[d]) {",
     "while (used[d] + run_act + need + 1 > w->dev_cap_mib[d]) {"),
    ("snapshot memory ignored", "if ((res[d] >> m) & 1u) used[d] += w->model_mib[m];",
     "if ((res[d] >> m) & 1u) used[d] += 0;"),
    ("device free after head only", "sf[ks] = s;", "sf[ks] = finish[h];"),
    ("completion from first arrival", "comp[wf] -= w->wf_arrival_us[wf];", "comp[wf] -= min_arr;"),
    ("headroom maximum", "< headroom) headroom", "> headroom) headroom"),
    ("load ignores the slot", "int64_t ls = t;", "int64_t ls = miss && pf[h] ? w->wf_arrival_us[wf] : r;"),
    ("pred finish ignored", "r = max64(r, finish[w->pred_idx[k]]);", "r = max64(r, start[w->pred_idx[k]]);"),
    # ranking key (Eq. 12)
    ("ready ignores arrival", "w->pred_off[h] == w->pred_off[h + 1] && w->wf_arrival_us[wf] <= 0",
     "w->pred_off[h] == w->pred_off[h + 1]"),
    ("admitted ignores capacity", "if (ready && fits) {", "if (ready) {"),
    ("class ignored", "admitted[wf_class ? wf_class[wf] : 0] += 1;", "admitted[0] += 1;"),
    ("ready completion at start", "c_ready = max64(c_ready, s);", "c_ready = max64(c_ready, start[h]);"),
    ("timely prefetch strict", "if (!ready && pf[h] && le <= r) timely += 1;",
     "if (!ready && pf[h] && le < r) timely += 1;"),
    ("timely prefetch counts ready work", "if (!ready && pf[h] && le <= r) timely += 1;",
     "if (pf[h] && le <= r) timely += 1;"),
    ("every load a reload", "if ((reclaimed[d] >> m) & 1u) h_life += le - ls;", "h_life += le - ls;"),
    ("loading delay from release", "if (ready) h_life += s - max64(r, free_before);",
     "if (ready) h_life += s - r;"),
    ("loading delay of all work", "if (ready) h_life += s - max64(r, free_before);",
     "h_life += s - max64(r, free_before);"),
    # paper victim order (Sec. 3.5, reclamation)
    ("paper order ignores redundancy", "if (redx != redy) return redx > redy;", ""),
    ("paper order prefers kept copies elsewhere", "if (redx != redy) return redx > redy;",
     "if (redx != redy) return redx < redy;"),
    ("paper ratio inverted", "if (a != b) return a > b;", "if (a != b) return a < b;"),
    ("paper order ignores reload cost", "const int64_t a = distx * loady, b = disty * loadx;",
     "const int64_t a = distx, b = disty;"),
    ("paper order ignores next use", "key[q][1] = nu == ORC_NO_USE ? ORC_NO_USE : nu - dev_index[pos];",
     "key[q][1] = 1;"),
    ("redundancy from live residency", "if (e != d && ((res_level[e] >> mm[q]) & 1u)) red = 1;",
     "if (e != d && ((res[e] >> mm[q]) & 1u)) red = 1;"),
    ("next use not advanced", "next_use[d * M + m] = next_after[pos];", ""),
    ("paper order most recently used", "return lastx < lasty;", "return lastx > lasty;"),
    # batch limit (Eq. 11, replica batch limit)
    ("running units hold no memory", "run_act += run_mem[q];", ""),
    ("running units lease nothing", "leased |= 1ull << run_model[q];", ""),
    ("no wait for running units", "|| next_fin == INT64_MAX) break;", "|| 1) break;"),
    ("slot that frees last", "if (sf[k] < sf[ks]) ks = k;", "if (sf[k] > sf[ks]) ks = k;"),
    ("queue overtaking", "dispatched[d] = t;", ""),
    # reclaimed copies per unit, prefix commit (Algorithm 1, Prefix_t)
    ("reclaims not reported", "if (rec_row) rec_row[h] |= 1ull << victim;", ""),
    ("prefix counts events at time 0", "if (finish_us[i] > 0 && finish_us[i] < t)",
     "if (finish_us[i] >= 0 && finish_us[i] < t)"),
    ("prefix ignores load ends", "if (le > 0 && le < t) t = le;", ""),
    ("prefix load end without the load", "const int64_t le = load_start_us[i] + w->load_us[(int64_t)w->act_model[i] * D + dev[i]];",
     "const int64_t le = load_start_us[i];"),
    ("prefix ignores arrivals", "if (w->wf_arrival_us[f] > 0 && w->wf_arrival_us[f] < t) t = w->wf_arrival_us[f];", ""),
    ("prefix commits at the event", "const int grant = start_us[i] < t;", "const int grant = start_us[i] <= t;"),
    ("prefix reclaims follow the start", "const int64_t first = load_start_us[i] >= 0 ? load_start_us[i] : start_us[i];",
     "const int64_t first = start_us[i];"),
]


def _pin_checks():
    """A fast selection of the pin tests (closed forms, second formulation,
    paper examples, invariants, metamorphic relations, exhaustive search)."""
    checks = []
    checks += [lambda s=s: t_ind.test_random_windows(s) for s in range(12)]
    checks += [lambda s=s: t_ind.test_tight_capacity(s) for s in range(4)]
    checks += [t_ind.test_capacity_flag_seen]
    checks += [lambda s=s: t_prop.test_single_device_closed_form(s) for s in range(3)]
    checks += [lambda s=s: t_prop.test_contention_free_longest_path(s) for s in range(3)]
    checks += [lambda s=s: t_prop.test_bounds_and_invariants(s) for s in range(6)]
    checks += [lambda s=s: t_prop.test_prefetch_never_hurts(s) for s in range(3)]
    checks += [lambda s=s: t_prop.test_time_shift_and_relabel(s) for s in range(3)]
    checks += [t_prop.test_objective_is_fp32_of_integer_outputs, t_prop.test_p95_nearest_rank_against_numpy,
               t_prop.test_p95_nearest_rank_many_workflow_counts]
    checks += [lambda s=s: t_prop.test_exact_fit_boundary(s) for s in (-1, 0, 1)]
    checks += [t_pap.test_fig4_one_load_one_prefetch_shared_by_two_workflows,
               t_pap.test_qmsum_fused_chain_one_grant_one_replica]
    checks += [lambda s=s: t_bf.test_exhaustive(s) for s in range(2)]
    checks += [lambda k=k: t_search.test_philox_known_answers(*k) for k in t_search.KAT]
    checks += [t_search.test_one_mutation_decoded_site_by_site, t_search.test_ranges_are_independent_of_splitting]
    checks += [lambda n=n: t_search.test_candidate_structure(n) for n in (1, 4)]
    checks += [lambda n=n: t_phi.test_worked_examples(n) for n in ("phi_reload", "phi_prefetch", "phi_ready_prefetch")]
    checks += [lambda s=s: t_phi.test_phi_from_schedule(s) for s in range(6)]
    checks += [lambda s=s: t_phi.test_phi_invariants(s) for s in range(3)]
    checks += [lambda n=n: t_vic.test_worked_examples(n)
               for n in ("victim_order", "victim_order_chain", "victim_order_snapshot",
                         "victim_order_ties")]
    checks += [lambda s=s: t_vic.test_paper_order_is_belady_optimal_on_one_device(s) for s in range(40)]
    checks += [lambda n=n: t_batch.test_worked_examples(n) for n in ("batch_memory", "batch_lease")]
    checks += [lambda s=s: t_batch.test_contention_free_longest_path(s) for s in (0, 1, 2, 3, 5, 6)]
    checks += [lambda s=s: t_batch.test_schedule_invariants(s) for s in range(8)]
    checks += [t_rep.test_worked_example, t_rep.test_both_outcomes_occur]
    checks += [lambda s=s: t_rep.test_cap_is_a_check_only(s) for s in range(3)]
    checks += [t_prefix.test_worked_example]
    checks += [t_rules.test_worked_example, t_rules.test_config_windows]
    checks += [lambda s=s: t_rules.test_against_second_formulation(s) for s in range(4)]
    checks += [lambda s=s: t_prefix.test_single_device_chain(s) for s in range(4)]
    checks += [lambda s=s: t_prefix.test_invariants(s) for s in range(4)]
    return checks


@pytest.fixture(scope="module")
def tmpdir_mod():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def test_unmutated_copy_passes(tmpdir_mod, monkeypatch):
    src = open(oracle.SRC_PATH).read()
    path = os.path.join(tmpdir_mod, "same.c")
    open(path, "w").write(src)
    lib = oracle.build(src=path, out=os.path.join(tmpdir_mod, "libsame.so"))
    monkeypatch.setattr(oracle, "LIB_PATH", lib)
    for check in _pin_checks():
        check()


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_killed(name, orig, mut, tmpdir_mod, monkeypatch):
    src = open(oracle.SRC_PATH).read()
    assert src.count(orig) == 1, f"fragment for '{name}' not found exactly once"
    tag = "".join(ch if ch.isalnum() else "_" for ch in name)
    path = os.path.join(tmpdir_mod, tag + ".c")
    open(path, "w").write(src.replace(orig, mut))
    lib = oracle.build(src=path, out=os.path.join(tmpdir_mod, "lib" + tag + ".so"))
    monkeypatch.setattr(oracle, "LIB_PATH", lib)
    for check in _pin_checks():
        try:
            with np.errstate(all="ignore"):
                check()
        except (AssertionError, oracle.OracleError, IndexError, ValueError, KeyError):
            return  # killed
    pytest.fail(f"mutant '{name}' survived every pin")
