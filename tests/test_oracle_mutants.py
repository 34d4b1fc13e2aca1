"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of oracle/oracle.c (on the CPU, in a
temporary directory), builds it with gcc, and runs every pin of
tests/test_oracle.py against that build: at least one pin must fail.
"""
import inspect
import os
import subprocess

import pytest

import goldens
import oracle
import test_oracle

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, original text, planted mistake)
MUTANTS = [
    ("id-before-ready", "if (w->ready[a] != w->ready[b]) return w->ready[a] < w->ready[b];\n"
                        "  int32_t pa",
     "int32_t pa"),
    ("ignore-priority", "if (pa != pb) return pa < pb;", ""),
    ("ready-tie-by-higher-id", "return a < b;\n}", "return a > b;\n}"),
    ("ignore-device-busy", "int64_t start = w->ready[v] > avail ? w->ready[v] : avail;",
     "int64_t start = w->ready[v];"),
    ("ignore-inputs", "int64_t start = w->ready[v] > avail ? w->ready[v] : avail;",
     "int64_t start = avail;"),
    ("min-instead-of-max", "if (out > w->ready[x]) w->ready[x] = out;",
     "if (out < w->ready[x] || w->ready[x] == 0) w->ready[x] = out;"),
    ("ready-on-first-pred", "if (--w->cnt[x] == 0) heap_push(g, w, x);",
     "if (w->cnt[x]-- == g->indeg[x]) heap_push(g, w, x);"),
    ("makespan-of-device-0", "for (int32_t r = 0; r < g->nres; ++r)\n        if (w->rfree[r] > span)",
     "for (int32_t r = 0; r < 1; ++r)\n        if (w->rfree[r] > span)"),
    ("placement-ignored", "int32_t r = J->place ? (int32_t)J->place[(int64_t)v * J->ld_place + s] : g->res[v];",
     "int32_t r = g->res[v];"),
    ("overflow-wraps", "if (f > INT32_MAX) {", "if (0) {"),
    ("accepts-zero-duration", "if (J->dur[(int64_t)v * J->ld_dur + s] < 1) st |= ORC_ST_BAD_DUR;",
     "if (J->dur[(int64_t)v * J->ld_dur + s] < 0) st |= ORC_ST_BAD_DUR;"),
    ("cp-drops-own-duration", "dist[v] = best[v] + d;", "dist[v] = best[v] + (best[v] ? 0 : d);"),
    ("cp-path-highest-id", "if (dist[p] == want && (nxt < 0 || p < nxt)) nxt = p;",
     "if (dist[p] == want && (nxt < 0 || p > nxt)) nxt = p;"),
    ("cp-end-highest-id", "if (dist[x] > dist[v]) v = x;", "if (dist[x] >= dist[v]) v = x;"),
    ("cycle-undetected", "return tail == g->n;", "return 1;"),
    ("static-ignores-device-order", "if (nx >= 0 && fin[v] > ready[nx]) ready[nx] = fin[v];", ""),
    ("static-ignores-inputs", "if (fin[v] > ready[g->si[e]]) ready[g->si[e]] = fin[v];", "(void)0;"),
    ("static-device-edges-reversed", "if (last_on_dev[r] >= 0) next_on_dev[last_on_dev[r]] = v;",
     "if (last_on_dev[r] >= 0) next_on_dev[v] = last_on_dev[r];"),
    ("static-accepts-repeats", "if (v < 0 || v >= n_ops || seen[v]) rc = ORC_E_INVAL;",
     "if (v < 0 || v >= n_ops) rc = ORC_E_INVAL;"),
    ("static-cycle-undetected", "if (tail != n_ops) rc = ORC_E_CYCLE;", "if (tail != n_ops) n_scen = 0;"),
    ("static-overflow-wraps", "if (fin[v] > INT32_MAX) {", "if (0) {"),
    ("attr-highest-id-pred", "if (w->fin[p] == start && (nxt < 0 || p < nxt)) nxt = p;",
     "if (w->fin[p] == start && (nxt < 0 || p > nxt)) nxt = p;"),
    ("attr-device-first", "v = nxt >= 0 ? nxt : w->prev[v];", "v = w->prev[v] >= 0 ? w->prev[v] : nxt;"),
    ("attr-end-highest-id", "if (w->fin[v] > w->fin[last]) last = v;", "if (w->fin[v] >= w->fin[last]) last = v;"),
    ("attr-busy-overwrites", "busy_r = A->busy[(int64_t)r * A->ld_res + s] + J->dur[(int64_t)v * J->ld_dur + s];",
     "busy_r = J->dur[(int64_t)v * J->ld_dur + s];"),
    ("attr-chain-stops-early", "if (start == 0) break;", "if (start <= d) break;"),
    ("attr-prev-not-recorded", "w->prev[v] = w->last[r];", "w->prev[v] = -1;"),
    ("philox-multipliers-swapped", "uint64_t p0 = (uint64_t)0xD2511F53u * x0;\n    uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;",
     "uint64_t p0 = (uint64_t)0xCD9E8D57u * x0;\n    uint64_t p1 = (uint64_t)0xD2511F53u * x2;"),
    ("philox-key-not-bumped", "    k1 += 0xBB67AE85u;\n", ""),
    ("philox64-words-crossed", "uint64_t y0 = (uint64_t)(p1 >> 64) ^ x1 ^ k0;", "uint64_t y0 = (uint64_t)(p0 >> 64) ^ x1 ^ k0;"),
    ("gen-drops-high-halves", "U += (int64_t)(x[i] & 0xFFFFu) + (int64_t)(x[i] >> 16);", "U += 2 * (int64_t)(x[i] & 0xFFFFu);"),
    ("gen-truncates-not-rounds", "int64_t adj = (q + ((int64_t)1 << 39)) >> 40;", "int64_t adj = q >> 40;"),
    ("gen-counter-words-swapped", "uint32_t ctr[4] = {(uint32_t)S, (uint32_t)((uint64_t)S >> 32), (uint32_t)v, 0};",
     "uint32_t ctr[4] = {(uint32_t)S, (uint32_t)v, (uint32_t)((uint64_t)S >> 32), 0};"),
    ("gen-knob-off-by-one", "int64_t k = (S / knob_block) % n_knobs;", "int64_t k = ((S + 1) / knob_block) % n_knobs;"),
    ("gen-local-scenario-index", "gen_one(J->base, J->n, J->n_knobs, J->knob_block, J->noise, J->seed, J->scen0 + s, v);",
     "gen_one(J->base, J->n, J->n_knobs, J->knob_block, J->noise, J->seed, s, v);"),
    ("gap-before-first-op", "if (J->gap && w->nrun[r] > 0) avail += J->gap[r];", "if (J->gap) avail += J->gap[r];"),
    ("gap-ignored", "if (J->gap && w->nrun[r] > 0) avail += J->gap[r];", "(void)0;"),
    ("gap-of-device-0", "if (J->gap && w->nrun[r] > 0) avail += J->gap[r];",
     "if (J->gap && w->nrun[r] > 0) avail += J->gap[0];"),
    ("gap-counted-in-makespan", "      w->rfree[r] = f;\n      if (J->gap) w->nrun[r]++;",
     "      w->rfree[r] = f + (J->gap && w->nrun[r] > 0 ? 0 : 0) + (J->gap ? J->gap[r] : 0);\n      if (J->gap) w->nrun[r]++;"),
    ("delay-of-device-0", "const int64_t out = J->delay ? f + J->delay[r] : f;",
     "const int64_t out = J->delay ? f + J->delay[0] : f;"),
    ("delay-ignored", "const int64_t out = J->delay ? f + J->delay[r] : f;", "const int64_t out = f;"),
    ("delay-holds-device", "      w->rfree[r] = f;\n      if (J->gap) w->nrun[r]++;",
     "      w->rfree[r] = J->delay ? f + J->delay[r] : f;\n      if (J->gap) w->nrun[r]++;"),
    ("gen-accepts-large-base", "if (b < 1 || b > ((int64_t)1 << 24)) return 0;", "if (b < 1) return 0;"),
    # bandwidth sharing
    ("share-ignores-count", "L->vt += (uint64_t)(t - L->tl) * (ORC_SHARE_UNIT / (uint64_t)L->k);",
     "L->vt += (uint64_t)(t - L->tl) * ORC_SHARE_UNIT;"),
    ("share-finish-one-ns-late", "return L->tl + (int64_t)((m - L->vt + per_ns - 1) / per_ns);",
     "return L->tl + (int64_t)((m - L->vt + per_ns) / per_ns);"),
    ("share-no-advance-on-arrival", "link_advance(L, w->ready[v]);\n        L->op[L->k] = v;",
     "L->op[L->k] = v;"),
    ("share-ops-before-finishes-on-ties", "lt <= w->ready[w->heap[0]]", "lt < w->ready[w->heap[0]]"),
    ("share-limit-off-by-one", "if (L->k == ORC_SHARE_MAX) {", "if (L->k == ORC_SHARE_MAX - 1) {"),
    ("share-accepts-zero-duration", "if (dv < 1) st |= ORC_ST_BAD_DUR;", "if (dv < 0) st |= ORC_ST_BAD_DUR;"),
    ("share-ready-on-first-pred", "w->cnt[x] -= 1;\n    if (w->cnt[x] == 0) heap_push(g, w, x);",
     "if (w->cnt[x]-- == g->indeg[x]) heap_push(g, w, x);"),
    ("share-overflow-wraps", "if (f > (int64_t)INT32_MAX) {", "if (0) {"),
    ("share-link-overflow-wraps", "if (lt > INT32_MAX) {", "if (0) {"),
    # the per-ns share of k active ops rounded other than down (a tuple
    # plants the same mistake at every listed site)
    ("share-ceil", ("L->vt += (uint64_t)(t - L->tl) * (ORC_SHARE_UNIT / (uint64_t)L->k);",
                    "const uint64_t per_ns = ORC_SHARE_UNIT / (uint64_t)L->k;"),
     ("L->vt += (uint64_t)(t - L->tl) * ((ORC_SHARE_UNIT + (uint64_t)L->k - 1) / (uint64_t)L->k);",
      "const uint64_t per_ns = (ORC_SHARE_UNIT + (uint64_t)L->k - 1) / (uint64_t)L->k;")),
    ("share-nearest", ("L->vt += (uint64_t)(t - L->tl) * (ORC_SHARE_UNIT / (uint64_t)L->k);",
                       "const uint64_t per_ns = ORC_SHARE_UNIT / (uint64_t)L->k;"),
     ("L->vt += (uint64_t)(t - L->tl) * ((ORC_SHARE_UNIT + (uint64_t)L->k / 2) / (uint64_t)L->k);",
      "const uint64_t per_ns = (ORC_SHARE_UNIT + (uint64_t)L->k / 2) / (uint64_t)L->k;")),
    # (a share rounded up only where the next finish is predicted is not a
    # mistake: the prediction is then early, nothing leaves at it, and the
    # replay predicts again from there, reaching the same finish times)
    ("share-ceil-in-advance-only", "L->vt += (uint64_t)(t - L->tl) * (ORC_SHARE_UNIT / (uint64_t)L->k);",
     "L->vt += (uint64_t)(t - L->tl) * ((ORC_SHARE_UNIT + (uint64_t)L->k - 1) / (uint64_t)L->k);"),
    ("share-exact-unit-need", "L->need[L->k] = L->vt + (uint64_t)d * ORC_SHARE_UNIT;",
     "L->need[L->k] = L->vt + (uint64_t)d * (ORC_SHARE_UNIT / 17 * 17);"),
]


def pins():
    for name, fn in inspect.getmembers(test_oracle, inspect.isfunction):
        if not name.startswith("test_"):
            continue
        if "g" in inspect.signature(fn).parameters:
            for g in goldens.all_goldens():
                yield f"{name}[{g['name']}]", (lambda fn=fn, g=g: lambda L: fn(g=g, library=L))()
        else:
            yield name, (lambda fn=fn: lambda L: fn(library=L))()


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, orig, mut):
    src = open(SRC).read()
    sites = zip(orig, mut) if isinstance(orig, tuple) else [(orig, mut)]
    for o, m in sites:
        assert src.count(o) == 1, f"mutation site of {name} not found"
        src = src.replace(o, m)
    path = tmp_path / "mutant.c"
    path.write_text(src)
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread",
                           "-I", os.path.dirname(SRC), str(path), "-o", str(so)])
    L = oracle.lib(str(so))
    caught = []
    for pin_name, pin in pins():
        try:
            pin(L)
        except (Exception, pytest.fail.Exception) as e:  # a failing pin
            caught.append((pin_name, type(e).__name__))
            break
    assert caught, f"no pin catches mutant {name}"
