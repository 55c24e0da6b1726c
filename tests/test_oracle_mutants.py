"""The pins catch plausible mistakes. Each case plants one mistake in a copy
of the oracle's C source (on the CPU only), builds it, and runs the pin
tests of that part of the path against it in a fresh process: at least one
pin must fail. The unmodified oracle passes the same pins elsewhere in this
suite."""
import concurrent.futures
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name, exact source text, replacement, pin files that must catch it
MUTANTS = [
    ("stats counts the diagonal", "if (a != b) coact[", "if (1) coact[",
     ["test_oracle_stats.py"]),
    ("stats keeps only the upper triangle", "if (a != b) coact[", "if (a < b) coact[",
     ["test_oracle_stats.py"]),
    ("SplitMix64 increment off by two", "z += 0x9e3779b97f4a7c15ULL;",
     "z += 0x9e3779b97f4a7c17ULL;", ["test_oracle_rng.py"]),
    ("bf16 ties round away from zero", "(lower == 0x8000u && (upper & 1u))",
     "(lower == 0x8000u)", ["test_oracle_bf16.py"]),
    ("Algorithm 1 keeps the last minimum cover",
     "if (covers) { bstar = b; found = 1; }", "if (covers) { bstar = b; }",
     ["test_oracle_assign.py"]),
    ("Algorithm 1 skips covers of one node", "for (int32_t size = 1; !found",
     "for (int32_t size = 2; !found", ["test_oracle_assign.py"]),
    ("Algorithm 1 tries sets by value before size",
     "                if (popcount32(b) != size) continue;\n", "", ["test_oracle_assign.py"]),
    ("remote mask keeps the home node's bit", "        if (n == home) continue;\n",
     "", ["test_oracle_assign.py"]),
    ("owner-only V counts the home node", "if (r / g != home) nodes |= 1u << (r / g);",
     "nodes |= 1u << (r / g);", ["test_oracle_assign.py"]),
    ("dispatch buckets transposed", "int64_t b = (int64_t)s * G + assigned[p];",
     "int64_t b = (int64_t)assigned[p] * G + s;", ["test_oracle_dispatch.py"]),
    ("dispatch offsets inclusive", "        offsets[b] = run;\n        run += counts[b];\n    }\n    offsets[GG] = run;",
     "        run += counts[b];\n        offsets[b] = run;\n    }\n    offsets[GG] = run;",
     ["test_oracle_dispatch.py"]),
    ("combine drops the last slot",
     "            for (int32_t j = 0; j < K; ++j) {\n                int64_t row = pos[t * K + j];",
     "            for (int32_t j = 0; j + 1 < K; ++j) {\n                int64_t row = pos[t * K + j];",
     ["test_oracle_combine.py"]),
    ("traffic V counts the home node", "            if (r / g != home) {\n                nodes |= 1u << (r / g);\n                *cross_pairs += 1;\n            }",
     "            nodes |= 1u << (r / g);\n            if (r / g != home) *cross_pairs += 1;",
     ["test_oracle_assign.py"]),
    ("node layout drops the source's own node", "                if (!mask[n]) {\n                    node_pos[t * N + n] = -1;",
     "                if (!mask[n] || n == s / g) {\n                    node_pos[t * N + n] = -1;",
     ["test_oracle_node_dispatch.py"]),
    ("forwarding mask uses global rank bits", "                mask[r / g] |= 1u << (r % g);\n            }\n            for (int32_t n = 0; n < N; ++n) {\n                if (!mask[n]) {",
     "                mask[r / g] |= 1u << (r % 32);\n            }\n            for (int32_t n = 0; n < N; ++n) {\n                if (!mask[n]) {",
     ["test_oracle_node_dispatch.py"]),
    ("node combine sums the partials in decreasing node order",
     "            for (int32_t n = 0; n < N; ++n) {\n                int64_t nrow = node_pos[t * N + n];\n                if (nrow < 0 || nrow >= node_rows) continue;\n                acc = acc + ",
     "            for (int32_t n = N - 1; n >= 0; --n) {\n                int64_t nrow = node_pos[t * N + n];\n                if (nrow < 0 || nrow >= node_rows) continue;\n                acc = acc + ",
     ["test_oracle_node_combine.py"]),
    ("node combine takes the node of a rank as r % g",
     "if (r < 0 || r >= G || r / g != n) continue;", "if (r < 0 || r >= G || r % g != n) continue;",
     ["test_oracle_node_combine.py"]),
    ("node combine drops the gate",
     "acc = fmaf(gates[t * K + j], ref_bf16_to_f32(expert_out[row * d + c]), acc);\n                }\n                partial[",
     "acc = acc + ref_bf16_to_f32(expert_out[row * d + c]);\n                }\n                partial[",
     ["test_oracle_node_combine.py"]),
    ("node combine truncates the partials",
     "partial[nrow * d + c] = ref_f32_to_bf16(acc);",
     "{ union { float f; uint32_t u; } cv; cv.f = acc; partial[nrow * d + c] = (uint16_t)(cv.u >> 16); }",
     ["test_oracle_node_combine.py"]),
    ("EMA weights swapped", "ema[i] = fmaf(decay, ema[i], gain * x);",
     "ema[i] = fmaf(gain, ema[i], decay * x);", ["test_oracle_ema.py"]),
    ("Ochiai diagonal left at zero", "uint32_t c = i == j ? count[i] : coact[(int64_t)i * E + j];",
     "uint32_t c = coact[(int64_t)i * E + j];", ["test_oracle_ema.py"]),
    ("Ochiai without the square root", "o = (float)c / sqrtf((float)count[i] * (float)count[j]);",
     "o = (float)c / ((float)count[i] * (float)count[j]);", ["test_oracle_ema.py"]),
    ("replica load indexed [G][E]", "load[(int64_t)e * G + r] += 1u;",
     "load[(int64_t)r * E + e] += 1u;", ["test_oracle_rebalance.py"]),
    ("Stage 2 places the lightest replica first",
     "    if (a->load != b->load) return a->load > b->load;\n    if (a->e != b->e) return a->e < b->e;\n    return a->r < b->r;",
     "    if (a->load != b->load) return a->load < b->load;\n    if (a->e != b->e) return a->e < b->e;\n    return a->r < b->r;",
     ["test_oracle_rebalance.py"]),
    ("Stage 1 objective counts each pair twice",
     "if (on[(int64_t)i * N + n] && on[(int64_t)j * N + n]) obj += q[(int64_t)i * E + j];",
     "if (on[(int64_t)i * N + n] && on[(int64_t)j * N + n]) obj += 2 * q[(int64_t)i * E + j];",
     ["test_oracle_plan.py"]),
    ("Stage 1 ignores the work cap in the local search",
     "                if (!(wna <= node_cap || wna <= work[na])) continue;",
     "", ["test_oracle_plan.py"]),
    ("Stage 1 skips the repair across nodes",
     "for (int64_t moves = 0; moves < 4 * (int64_t)G * S; ++moves) {",
     "for (int64_t moves = 0; moves < 0; ++moves) {", ["test_oracle_plan.py"]),
    ("exact Stage 1 counts a node's pairs on its first rank only",
     "for (int32_t i = 0; i < x->g; ++i) on |= x->cur[n * x->g + i];",
     "on = x->cur[n * x->g];", ["test_oracle_plan_exact.py"]),
    ("exact Stage 1 ignores the work cap", "        if (!exact_divisible(x)) return;\n",
     "", ["test_oracle_plan_exact.py"]),
    ("exact Stage 1 needs every expert of a set on one rank",
     "if (x->cur[r] & A) ++holders;", "if ((x->cur[r] & A) == A) ++holders;",
     ["test_oracle_plan_exact.py"]),
    ("exact Stage 1 allows one slot fewer", "if (popcount32(m) > x->S) continue;",
     "if (popcount32(m) >= x->S) continue;", ["test_oracle_plan_exact.py"]),
    ("exact Stage 1 keeps the last best layout", "if (x->found && !(v > x->best)) return;",
     "if (x->found && !(v >= x->best)) return;", ["test_oracle_plan_exact.py"]),
    ("Stage 1 skips the retries with node slack",
     "for (int k = 0; k < 3 && !ok; ++k) {", "for (int k = 0; k < 0 && !ok; ++k) {",
     ["test_oracle_plan_milp.py"]),
]


def _run(case, tmp):
    name, old, new, pins = case
    src = open(oracle.SRC_PATH).read()
    assert src.count(old) >= 1, f"{name}: source text not found"
    slug = "".join(c if c.isalnum() else "_" for c in name)
    c_path = os.path.join(tmp, slug + ".c")
    so_path = os.path.join(tmp, slug + ".so")
    with open(c_path, "w") as f:
        f.write(src.replace(old, new, 1))
    subprocess.run(["gcc", *oracle.CFLAGS, c_path, "-o", so_path, "-lm"], check=True)
    env = dict(os.environ, ORACLE_LIB=so_path)
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
           *[os.path.join(ROOT, "tests", p) for p in pins]]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode, r.stdout[-400:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda c: _run(c, str(tmp_path)), MUTANTS))
    survived = [(n, out) for n, rc, out in results if rc == 0]
    assert not survived, f"mistakes no pin caught: {survived}"
    # a pytest failure (1), not a crash of the runner (e.g. 2 or 4)
    assert all(rc == 1 for _, rc, _ in results), [(n, rc) for n, rc, _ in results]
