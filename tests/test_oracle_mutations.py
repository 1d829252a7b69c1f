"""The oracle's pins have teeth: plausible mistakes planted in a copy of the
oracle source (on the CPU only) must each fail at least one pin.

Each mutation is a text substitution on ``oracle/mts_oracle.c``; the mutated
copy is compiled to a temporary library and the pin suites run against it in
a subprocess.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "mts_oracle.c")

MUTATIONS = {
    # Eq. 4: headroom charged per running request instead of once per tier
    "headroom_per_request": [("present[sl[s].tier] = 1;", "present[sl[s].tier] += 1;"),
                             ("if (present[p]) v256 += rp->hq[p];",
                              "v256 += present[p] * rp->hq[p];")],
    # Eq. 2: head-of-line demand with the wrong sign
    "hol_sign": [("int64_t v256 = 256 * (phys + demand);", "int64_t v256 = 256 * (phys - demand);")],
    # Section 3.4: ties in F go to the highest index
    "dispatch_tie": [("if (best < 0 || f_greater(num[i], den[i], num[best], den[best])) best = (int)i;",
                      "if (best < 0 || !f_greater(num[best], den[best], num[i], den[i])) best = (int)i;")],
    # Section 3.4: lowest tier first instead of tier 0 first
    "dispatch_order": [("for (uint32_t p = 0; p < (x->cfg.tier_blind ? 1 : K); ++p) {\n        for (uint32_t k = 0; k < n; ++k) {",
                        "for (uint32_t p = (x->cfg.tier_blind ? 1 : K); p-- > 0;) {\n        for (uint32_t k = 0; k < n; ++k) {")],
    # Eq. 3 reading: the lowest tier keeps its headroom
    "lowest_tier_headroom": [("if (c->zero_lowest) out[K - 1] = 0;", "")],
    # preemption takes the oldest instead of the newest request of the worst tier
    "preempt_order": [("if (ps > pv || (ps == pv && sl[s].seq > sl[v].seq)) v = (int)s;",
                       "if (ps > pv || (ps == pv && sl[s].seq < sl[v].seq)) v = (int)s;")],
    # KV growth one token late
    "growth_off_by_one": [("if (sl[s].st == ST_RUNNING && sl[s].len % blk == 0) grow++;",
                           "if (sl[s].st == ST_RUNNING && (sl[s].len + 1) % blk == 0) grow++;")],
    # Section 3.5: strict instead of non-strict theta threshold
    "theta_strict": [("if (lhs < rhs) break;", "if (lhs <= rhs) break;")],
    # Poisson recursion with a wrong index
    "poisson_index": [("p = p * c->arr_mean / (double)n;", "p = p * c->arr_mean / (double)(n + 1);")],
    # Philox multiplier typo
    "philox_constant": [("mulhilo64(0xD2E7470EE14C6C93ULL", "mulhilo64(0xD2E7470EE14C6C95ULL")],
    # migration candidate: largest instead of smallest KV footprint
    "candidate_footprint": [("(bs < bc || (bs == bc && sl[s].seq > sl[c].seq))",
                             "(bs > bc || (bs == bc && sl[s].seq > sl[c].seq))")],
    # staged copy: commit one stage early
    "commit_early": [("if (m->copied < b) continue;", "if (m->copied + 1 < b) continue;")],
    # Section 3.4: a draining instance still takes dispatches
    "drain_dispatchable": [("if (nempty[i] == 0 || rp->drain[i]) continue;", "if (nempty[i] == 0) continue;")],
    # Section 3.4: all-draining fallback picks the lowest index, not the least loaded
    "drain_fallback_first": [("if (best < 0 || f_greater(num[j], den[j], num[best], den[best])) best = (int)j;",
                              "if (best < 0) best = (int)j;")],
    # Section 3.5: a draining instance accepted as a migration destination
    "drain_destination": [("        if (rp->drain[dst]) break;\n", "")],
    # Section 3.4: F_normal charged with tier-0 headroom
    "fnormal_headroom": [("*num = 256 * ((int64_t)x->cfg.kv_blocks - phys - demand);",
                          "*num = 256 * ((int64_t)x->cfg.kv_blocks - phys - demand) - x->Hq[rp->group][0];")],
    # Section 3.6: scale-out at an average of exactly -0.5
    "scale_out_inclusive": [("if (acc < -half) return -1;", "if (acc <= -half) return -1;")],
    # latency histograms: sub-ranges of a quarter octave instead of an eighth
    "hist_quarter_octave": [("uint64_t sub = (v >> (e - 3)) - 8;  /* 0..7 */",
                             "uint64_t sub = ((v >> (e - 2)) - 4) * 2;  /* 0..7 */")],
    # latency histograms: queue delay counted again after every re-admission
    "hist_qdelay_every_admission": [
        ("                hist_add(rp, H_QDELAY, sl[h].tier, t - sl[h].tarr);\n            }",
         "            }\n            hist_add(rp, H_QDELAY, sl[h].tier, t - sl[h].tarr);")],
    # latency histograms: end-to-end time measured to the tick before the last token
    "hist_e2e_early": [("hist_add(rp, H_E2E, sl[s].tier, t - sl[s].tarr);",
                        "hist_add(rp, H_E2E, sl[s].tier, t - 1 - sl[s].tarr);")],
    # INFaaS: largest instead of smallest cost
    "infaas_argmax": [("if (best < 0 || c < bc) { best = (int)i; bc = c; }",
                       "if (best < 0 || c > bc) { best = (int)i; bc = c; }")],
    # INFaaS: ties go to the highest index
    "infaas_tie_high": [("if (best < 0 || c < bc) { best = (int)i; bc = c; }",
                         "if (best < 0 || c <= bc) { best = (int)i; bc = c; }")],
    # INFaaS: migration left on
    "infaas_migrates": [("if (t % x->cfg.mig_interval != 0 || x->cfg.policy == POLICY_INFAAS) return;",
                         "if (t % x->cfg.mig_interval != 0) return;")],
    # INFaaS: moving average rounded toward zero instead of down
    "infaas_ewma_trunc": [("rp->svc[i] += floor_shift(mean - rp->svc[i], x->cfg.ewma_shift);",
                           "rp->svc[i] += (mean - rp->svc[i]) / ((int64_t)1 << x->cfg.ewma_shift);")],
    # tier-blind scheduling that still orders queues by tier
    "blind_ignored": [("static uint32_t prio(const or_ctx *x, uint32_t tier) { return x->cfg.tier_blind ? 0 : tier; }",
                       "static uint32_t prio(const or_ctx *x, uint32_t tier) { (void)x; return tier; }")],
    # tier-blind scheduling that still dispatches tier 0 first
    "blind_dispatch_tier_order": [("    for (uint32_t p = 0; p < (x->cfg.tier_blind ? 1 : K); ++p) {",
                                   "    for (uint32_t p = 0; p < K; ++p) {"),
                                  ("            if (prio(x, a[0]) != p) continue;", "            if (a[0] != p) continue;")],
    # INFaaS: INTERFERED takes precedence over OVERLOADED
    "infaas_state_order": [("    if (h >= 0 && (int64_t)blocks(x, inst_slots(x, rp, i)[h].len) > rp->freeb[i]) return x->cfg.pen_over;\n    if (rp->intf[i]) return x->cfg.pen_intf;",
                            "    if (rp->intf[i]) return x->cfg.pen_intf;\n    if (h >= 0 && (int64_t)blocks(x, inst_slots(x, rp, i)[h].len) > rp->freeb[i]) return x->cfg.pen_over;")],
    # Section 6.5 promotion: strict instead of non-strict quota
    "promote_strict_age": [("if (c->promote_age[sl->tier] != 0 && age >= c->promote_age[sl->tier]) sl->tier -= 1;",
                            "if (c->promote_age[sl->tier] != 0 && age > c->promote_age[sl->tier]) sl->tier -= 1;")],
    # Section 6.5 promotion: two tiers per pass
    "promote_two_tiers": [("age >= c->promote_age[sl->tier]) sl->tier -= 1;",
                           "age >= c->promote_age[sl->tier]) sl->tier = sl->tier >= 2 ? sl->tier - 2 : 0;")],
    # Section 6.5 promotion: running requests promoted too
    "promote_running": [("if (sl->st != ST_WAITING || sl->tier == 0) continue;",
                         "if (sl->st == ST_EMPTY || sl->tier == 0) continue;")],
    # Section 6.5 adaptive headroom: a mean exactly on target counts as a miss
    "adapt_miss_inclusive": [("if (d > slo * a) h =", "if (d >= slo * a) h =")],
    # Section 6.5 adaptive headroom: the two steps swapped
    "adapt_steps_swapped": [("h = h + c->adapt_up > c->adapt_max ? c->adapt_max : h + c->adapt_up;",
                             "h = h + c->adapt_down > c->adapt_max ? c->adapt_max : h + c->adapt_down;"),
                            ("h = h < c->adapt_down ? 0 : h - c->adapt_down;",
                             "h = h < c->adapt_up ? 0 : h - c->adapt_up;")],
    # Section 6.5 adaptive headroom: the lowest tier adapts under zero_lowest
    "adapt_lowest_tier": [("if ((c->zero_lowest && p == K - 1) || a == 0) continue;", "if (a == 0) continue;")],
    # Section 4.4 workloads: prompt lengths drawn from the output table and output
    # lengths from the prompt table
    "length_tables_swapped": [
        ("a[1] = x->prompt_tab.base + sample(&x->prompt_tab, (uint32_t)r[1]);\n        a[2] = x->out_tab.base + sample(&x->out_tab, (uint32_t)r[2]);",
         "a[1] = x->out_tab.base + sample(&x->out_tab, (uint32_t)r[1]);\n        a[2] = x->prompt_tab.base + sample(&x->prompt_tab, (uint32_t)r[2]);")],
    # the output length drawn from the prompt's random word (correlated lengths)
    "length_shared_word": [("a[2] = x->out_tab.base + sample(&x->out_tab, (uint32_t)r[2]);",
                            "a[2] = x->out_tab.base + sample(&x->out_tab, (uint32_t)r[1]);")],
    # Section 6.5 adaptive headroom: counters never re-based (cumulative means)
    "adapt_cumulative": [("        rp->snap_adm[p] = adm;\n        rp->snap_qd[p] = qd;\n", "")],
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, tmp_path):
    src = open(SRC).read()
    for old, new in MUTATIONS[name]:
        assert src.count(old) == 1, "mutation anchor not found exactly once: %r" % old
        src = src.replace(old, new)
    cfile = tmp_path / "mutant.c"
    cfile.write_text(src)
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                           "-o", str(lib), str(cfile), "-lm"])
    env = dict(os.environ, MTS_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_sampling_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_drain_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_hist_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_infaas_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_exact.py"),
                        os.path.join(ROOT, "tests", "test_oracle_adaptive_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, "mutation %s survived every pin:\n%s" % (name, r.stdout[-2000:])
