"""Each plausible mistake planted in a copy of the oracle makes at least one
pin fail.  The copy is compiled into a temporary library and the pins run in
a subprocess that loads it; the committed oracle is never modified."""
import os
import subprocess
import sys

import pytest

from oracle import build as oracle_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

CACHE = ["tests/test_oracle_cache.py", "tests/test_oracle_replay.py"]
PRIM = ["tests/test_oracle_primitives.py"]
METRIC = ["tests/test_oracle_metrics.py", "tests/test_oracle_replay.py"]
POLICY = ["tests/test_oracle_policies.py"]
CONC = ["tests/test_oracle_concentration.py"]
GATES = ["tests/test_oracle_gates.py"]
ARENA = ["tests/test_oracle_arena.py"]

# (name, source text, replacement, pins expected to catch it)
MISTAKES = [
    ("refinement replaces on equal score", "sST[rest[nrep]] > sST[weakest[nrep]]",
     "sST[rest[nrep]] >= sST[weakest[nrep]]", CACHE),
    ("lowest-priority ranking takes the higher index on ties", "(best < 0 || s[u] < s[best])) best = u;",
     "(best < 0 || s[u] <= s[best])) best = u;", CACHE),
    ("refinement score drops p^S", "sST[e] = aT[e] + pred[e];", "sST[e] = aT[e];", CACHE),
    ("retention score drops p^R", "sT[e] = pR[e] + pT[e];", "sT[e] = pT[e];", CACHE),
    ("selected experts not protected", "leavable[u] = (uint8_t)(C[u] && !sel[u]);", "leavable[u] = C[u];", CACHE),
    ("refinement at the first token", "if (spatio && t >= 1 && c->R > 0) {", "if (spatio && t >= 0 && c->R > 0) {",
     CACHE),
    ("silu sign", "act[f] = a / (1.0 + exp(-a)) * b;", "act[f] = a / (1.0 + exp(a)) * b;", PRIM),
    ("Cody-Waite low part dropped", "r = fmaf(-k, g_ln2_lo, r);", "r = r;", PRIM),
    ("warm-up boundary off by one", "const int counted = t >= c->warmup_tokens;",
     "const int counted = t > c->warmup_tokens;", METRIC),
    ("LRU clock not advanced", "if (selected[e]) pol[e] = (float)(2 * t + 2);", "pol[e] = pol[e];", POLICY),
    ("LFU counts unselected experts", "if (selected[e]) pol[e] = pol[e] + 1.0f;", "pol[e] = pol[e] + 1.0f;", POLICY),
    ("LRFU without decay", "float v = pol[e] * w;", "float v = pol[e];", POLICY),
    ("Spatio-only keeps s^T as its a-score", "c->mode == ORC_MODE_SPATIO_ONLY ? pR : sT", "sT", POLICY),
    ("proactive insertion not stamped", "for (int i = 0; i < nP; ++i) st->pol[sl * N + loaded[i]] = (float)(2 * t + 1);",
     ";", POLICY),
    ("proactive insertion stamped as an access",
     "st->pol[sl * N + loaded[i]] = (float)(2 * t + 1);", "st->pol[sl * N + loaded[i]] = (float)(2 * t + 2);", POLICY),
    ("LRFU weight with the wrong sign", "return (float)pow(2.0, -(double)lambda);",
     "return (float)pow(2.0, (double)lambda - 1.0);", POLICY),
    ("entropy in bits", "if (f[e] > 0.0) H -= f[e] * log(f[e]);", "if (f[e] > 0.0) H -= f[e] * log2(f[e]);", CONC),
    ("effective experts as entropy", "        acc[0] += exp(H);", "        acc[0] += H;", CONC),
    ("top-m mass takes one too many", "for (int i = 0; i < top_m && i < N; ++i) {",
     "for (int i = 0; i <= top_m && i < N; ++i) {", CONC),
    ("selection counts drop one expert", "for (int k = 0; k < K; ++k) st->selcount[(size_t)l * N + sel[k]] += 1;",
     "for (int k = 0; k < K - 1; ++k) st->selcount[(size_t)l * N + sel[k]] += 1;", CONC),
    ("highest free slot first", "for (int q = 0; q < st->n_slots; ++q) {",
     "for (int q = st->n_slots - 1; q >= 0; --q) {", ["tests/test_oracle_replay.py"]),
    ("softmax without the max shift", "float diff = z[e] - m;", "float diff = z[e];", PRIM),
    ("Top-K prefers the higher index on ties", "if (best < 0 || v[e] > v[best]) best = e;",
     "if (best < 0 || v[e] >= v[best]) best = e;", PRIM),
    ("native bias dropped", "if (bias) acc += (double)bias[e];", "if (bias) acc += 0.0;", PRIM),
    ("logits accumulated in fp32", "for (int i = 0; i < d; ++i) acc += (double)w[i] * (double)h[i];",
     "for (int i = 0; i < d; ++i) acc = (float)(acc + (double)w[i] * (double)h[i]);", PRIM),
    ("gates not renormalised", "out->gate[sl * K + k] = (double)pR[sel[k]] / gsum;",
     "out->gate[sl * K + k] = (double)pR[sel[k]];", GATES),
    ("refinement examines candidates from the lowest score up", "if (!C[A[i]]) fresh[nfresh++] = A[i];",
     "if (!C[A[R - 1 - i]]) fresh[nfresh++] = A[R - 1 - i];", CACHE),
    ("refinement displaces without checking the next weakest", "while (nrep < nrest && nrep < nw && ",
     "while (nrep < nrest && nrep < nw && nrep < 1 && ", CACHE),
    ("retention evicts one too few", "const int surplus = orc_count(C, N) + nD - cap;",
     "const int surplus = orc_count(C, N) + nD - cap - 1;", CACHE),
    ("down projection transposed", "acc += (double)wd[(size_t)j * F + f] * act[f];",
     "acc += (double)wd[(size_t)f * d + j] * act[f];", PRIM),
    ("up projection reads the gate weights", "b += (double)wu[(size_t)f * d + i] * (double)x[i];",
     "b += (double)wg[(size_t)f * d + i] * (double)x[i];", PRIM),
    ("residents give up their slots", "if (slot[e] >= 0 && !inU[e]) slot[e] = -1;", "slot[e] = -1;",
     ["tests/test_oracle_replay.py"]),
    ("arena evicts the most recently used", "if (victim < 0 || stamp[v] < stamp[victim] ||",
     "if (victim < 0 || stamp[v] > stamp[victim] ||", ARENA),
    ("arena evicts the higher slot on equal recency", "(stamp[v] == stamp[victim] && slot[v] < slot[victim]))",
     "(stamp[v] == stamp[victim] && slot[v] > slot[victim]))", ARENA),
    # (evicting an expert only a later round needs is not a distinct mistake:
    # with resident experts executed first, no round that must evict has a
    # resident expert left for a later round)
    ("arena evicts an expert its own round needs", "if (slot[v] < 0 || round_of[v] >= r) continue;",
     "if (slot[v] < 0 || round_of[v] > r) continue;", ARENA),
    ("arena rounds start with the missing experts",
     "        if (E[e] && slot[e] >= 0) order[nE++] = e;\n    for (int e = 0; e < N; ++e)\n"
     "        if (E[e] && slot[e] < 0) order[nE++] = e;",
     "        if (E[e] && slot[e] < 0) order[nE++] = e;\n    for (int e = 0; e < N; ++e)\n"
     "        if (E[e] && slot[e] >= 0) order[nE++] = e;", ARENA),
    ("executed experts keep their old recency", "                if (E[e]) stamp[e] = now;",
     "                if (E[e]) stamp[e] = stamp[e];", ARENA),
    ("arena rounds leave recency unchanged", "for (int i = lo; i < hi; ++i) stamp[order[i]] = now;",
     "for (int i = lo; i < hi; ++i) stamp[order[i]] = stamp[order[i]];", ARENA),
]


@pytest.mark.parametrize("name,old,new,pins", MISTAKES, ids=[m[0] for m in MISTAKES])
def test_planted_mistake_is_caught(name, old, new, pins, tmp_path):
    src = open(SRC).read()
    assert src.count(old) == 1, f"the planted site moved: {old}"
    mutant = tmp_path / "oracle_mutant.c"
    mutant.write_text(src.replace(old, new))
    lib = oracle_build.compile_library(str(mutant), str(tmp_path / "liboracle_mutant.so"))
    env = dict(os.environ, ORACLE_LIBRARY=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *pins], cwd=ROOT,
                       env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"no pin caught: {name}\n{r.stdout[-2000:]}"
