"""The oracle's pins catch plausible mistakes (no GPU).

Each case compiles a copy of the oracle with one mistake planted in it. The
mistakes are a reversed order, a non-strict comparison, an index off by one,
a dropped or swapped term, or the wrong head or row. The case then runs the
pin module of that function (tests/test_oracle_<stage>.py) on the copy, in a
pytest subprocess that loads it through ORACLE_LIB; at least one pin must
fail. The unmodified source must pass every pin the same way. The RNN head
has its own file (test_oracle_rnn_mutants.py).
"""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
REPO = os.path.dirname(HERE)

SCHED, ATTN, ACC, DRAFT = (os.path.join(HERE, f"test_oracle_{m}.py")
                           for m in ("schedule", "attention", "accept", "draft"))

MUTANTS = {
    # ---- Algorithm 1
    "schedule: ascending admission order": (SCHED,
        "    if (p->a > q->a) return -1;\n    if (p->a < q->a) return 1;",
        "    if (p->a > q->a) return 1;\n    if (p->a < q->a) return -1;"),
    "schedule: equal throughput counts as a gain": (SCHED,
        "        if (theta > theta_best) {", "        if (theta >= theta_best) {"),
    "schedule: tau starts at zero": (SCHED,
        "    double tau = (double)R;", "    double tau = 0.0;"),
    "schedule: throughput read one batch size early": (SCHED,
        "        double theta = tau * sps[B];", "        double theta = tau * sps[B - 1];"),
    "schedule: exclusive survival product": (SCHED,
        "            p = p * c;\n            a[(int64_t)r * K + j] = p;",
        "            a[(int64_t)r * K + j] = p;\n            p = p * c;"),
    "schedule: mode 1 stops at the first loss as well": (SCHED,
        "        } else if (mode == 0) {\n            break;", "        } else {\n            break;"),
    "schedule: snapshot of the admitted request only": (SCHED,
        "            for (int r = 0; r < R; ++r) len[r] = l[r]; /* snapshot l* <- l */",
        "            len[E[i].r] = E[i].j;"),
    "schedule: margin in absolute throughput units": (SCHED,
        "        double m = fabs(theta - theta_best) / theta_best;",
        "        double m = fabs(theta - theta_best);"),
    "accept: draw margin not divided by the total mass": (ACC,
        "            double m1 = (thr - prev) / total, m2 = (cum - thr) / total;",
        "            double m1 = thr - prev, m2 = cum - thr;"),
    "schedule capacity: taken from the search with the early stop": (SCHED,
        "    int rc = oracle_schedule(conf_prev, R, K, sps, sps_len, 1, len, NULL, &n_adm,",
        "    int rc = oracle_schedule(conf_prev, R, K, sps, sps_len, 0, len, NULL, &n_adm,"),
    "schedule top-K: one candidate past the capacity": (SCHED,
        "    int64_t take = capacity < 0 ? 0 : (capacity < n ? capacity : n);",
        "    int64_t take = capacity < 0 ? 0 : (capacity + 1 < n ? capacity + 1 : n);"),
    "schedule top-K: ranked by the position's own confidence": (SCHED,
        "    oracle_survival(conf, R, K, a);\n    int64_t n = 0;",
        "    for (int64_t i = 0; i < (int64_t)R * K; ++i) a[i] = conf_value(conf[i]);\n"
        "    int64_t n = 0;"),
    "schedule top-K: the capacity is ignored": (SCHED,
        "    for (int64_t i = 0; i < take; ++i) len[E[i].r] = E[i].j;",
        "    for (int64_t i = 0; i < n; ++i) len[E[i].r] = E[i].j;"),
    # ---- verify attention
    "attention: causal limit one key short": (ATTN,
        "        int64_t visible = (int64_t)kv_len[r] - ql + t + 1;",
        "        int64_t visible = (int64_t)kv_len[r] - ql + t;"),
    "attention: KV head by modulo": (ATTN,
        "        int g = h / group;", "        int g = h % Hkv;"),
    "attention: scale dropped": (ATTN,
        "            s[j] = scale * dot;", "            s[j] = dot;"),
    "attention: unnormalised weights": (ATTN,
        "            double w = s[j] / den;", "            double w = s[j];"),
    "attention: lse without the maximum": (ATTN,
        "        if (lse) lse[i] = m + log(den);", "        if (lse) lse[i] = log(den);"),
    # ---- acceptance
    "accept: residual sign swapped": (ACC,
        "                        double e = p[v] - (double)pd[v];",
        "                        double e = (double)pd[v] - p[v];"),
    "accept: ratio inverted": (ACC,
        "                double ratio = pdx > 0.0 ? p[x] / pdx : INFINITY;",
        "                double ratio = p[x] > 0.0 ? pdx / p[x] : INFINITY;"),
    "accept: bonus from the last tested row": (ACC,
        "                const void* row = base + (size_t)(cu_q[r] + l) * (size_t)ld * esz;\n"
        "                target_dist(row, logit_dtype, V, inv_temp, p);\n                double cm;",
        "                const void* row = base + (size_t)(cu_q[r] + (l > 0 ? l - 1 : 0)) * (size_t)ld * esz;\n"
        "                target_dist(row, logit_dtype, V, inv_temp, p);\n                double cm;"),
    "accept: greedy ties go to the highest index": (ACC,
        "        if (x > bv) { bv = x; best = v; }", "        if (x >= bv) { bv = x; best = v; }"),
    "accept: rate sums the larger probability": (ACC,
        "ar += p[v] < (double)pd[v] ? p[v] : (double)pd[v];",
        "ar += p[v] > (double)pd[v] ? p[v] : (double)pd[v];"),
    "accept: inverse CDF takes the bucket edge": (ACC,
        "        if (cum > thr) {", "        if (cum >= thr) {"),
    "accept: test reads the next uniform": (ACC,
        "                double uu = (double)u[(int64_t)r * (K + 1) + t];",
        "                double uu = (double)u[(int64_t)r * (K + 1) + t + 1];"),
    "accept: greedy rejection emits the bonus row's argmax": (ACC,
        "                if (draft_tok[(int64_t)r * K + t] != am) { acc = t; tok = am; break; }",
        "                if (draft_tok[(int64_t)r * K + t] != am) { acc = t; tok = argmax_row("
        "base + (size_t)(cu_q[r] + l) * (size_t)ld * esz, logit_dtype, V); break; }"),
    # ---- Markov-head draft block
    "draft: embedding does not follow the draws": (DRAFT,
        "            prev = x;\n        }\n        free(z);\n        free(e);",
        "            (void)x;\n        }\n        free(z);\n        free(e);"),
    "draft: temperature outside the bias": (DRAFT,
        "                z[v] = inv_temp * (elem(U, row * ld + v, u_dtype) + b);",
        "                z[v] = inv_temp * elem(U, row * ld + v, u_dtype) + b;"),
    "draft: confidence temperature multiplies": (DRAFT,
        "            conf[row] = 1.0 / (1.0 + exp(-sacc / T));",
        "            conf[row] = 1.0 / (1.0 + exp(-sacc * T));"),
    "draft: draw uses the next position's uniform": (DRAFT,
        "            const int x = inverse_cdf(z, V, (double)u[row], &mg);",
        "            const int x = inverse_cdf(z, V, (double)u[(int64_t)r * K + (k % K)], &mg);"),
}


def _compile(text, d):
    src, lib = os.path.join(d, "oracle.c"), os.path.join(d, "liboracle.so")
    with open(src, "w") as f:
        f.write(text)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
                           "-fno-fast-math", "-shared", "-fPIC", src, "-o", lib, "-lm"])
    return lib


def _run_pins(lib, *modules):
    env = dict(os.environ, ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    return subprocess.run([sys.executable, "-m", "pytest", *modules, "-x", "-q", "-m", "not gpu",
                           "-p", "no:cacheprovider", "-p", "no:xdist"],
                          cwd=REPO, env=env, capture_output=True, text=True, timeout=600)


def _source():
    with open(oracle._SRC) as f:
        return f.read()


def test_unmodified_source_passes_every_pin(tmp_path):
    lib = _compile(_source(), str(tmp_path))
    r = _run_pins(lib, SCHED, ATTN, ACC, DRAFT)
    assert r.returncode == 0, r.stdout[-3000:]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name, tmp_path):
    module, old, new = MUTANTS[name]
    text = _source()
    assert text.count(old) == 1, f"mutation site for {name!r} not found once"
    lib = _compile(text.replace(old, new), str(tmp_path))
    r = _run_pins(lib, module)
    assert r.returncode != 0, f"no pin caught: {name}"
