"""The oracle's pins must catch plausible mistakes.

Each case below plants one mistake in a copy of oracle/oracle.cpp (a dropped
term, a wrong sign, index or operand, an off-by-one bound, a wrong rounding),
builds it on the CPU, and runs the pins of tests/test_oracle.py against that
build in a child process: at least one pin must fail (or the broken build
must crash).  The golden fixture is not used: it would flag any change, and
the point is that the checks written from the paper and the mathematics do.
"""
import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.cpp")
FLAGS = ["-O2", "-std=c++17", "-fno-fast-math", "-ffp-contract=off", "-shared", "-fPIC"]

FWD_LOOP = ("    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n"
            "      for (int e = 0; e < E; ++e) acc[e] += double(W.get(t, I[s], e));")

MUTATIONS = {
    # forward (Algorithm 1)
    "fwd_drops_last_lookup": (FWD_LOOP, FWD_LOOP.replace("s < O[k + 1]", "s < O[k + 1] - 1")),
    "fwd_wrong_table": ("    const int t = int(k / B);\n    std::fill(acc.begin(), acc.end(), 0.0);\n"
                        "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n      for",
                        "    const int t = int(k % T);\n    std::fill(acc.begin(), acc.end(), 0.0);\n"
                        "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n      for"),
    "fwd_fp32_accumulator": ("acc[e] += double(W.get(t, I[s], e));",
                             "acc[e] = double(float(acc[e]) + W.get(t, I[s], e));"),
    "fwd_no_reset_between_bags": ("    const int t = int(k / B);\n    std::fill(acc.begin(), acc.end(), 0.0);\n"
                                  "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n      for",
                                  "    const int t = int(k / B);\n"
                                  "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n      for"),
    "split_fwd_wrong_shift": ("return bits_to_float(uint32_t(hi[t][r * E + e]) << 16);",
                              "return bits_to_float(uint32_t(hi[t][r * E + e]) << 15);"),
    # dedup (keys, bags, stable sort, unique)
    "dedup_unstable_sort": ("std::stable_sort(perm.begin(), perm.end(),",
                            "std::sort(perm.begin(), perm.end(),"),
    "dedup_key_without_rowbase": ("d.key[s] = uint32_t(d.rowbase[k / B] + I[s]);",
                                  "d.key[s] = uint32_t(I[s]);"),
    "dedup_bag_within_table": ("d.bag[s] = uint32_t(k);", "d.bag[s] = uint32_t(k % B);"),
    "table_of_key_boundary": ("while (int64_t(key) >= d.rowbase[t + 1]) ++t;",
                              "while (int64_t(key) > d.rowbase[t + 1]) ++t;"),
    # update (Algorithms 2-4 fused)
    "update_wrong_sign": ("w[e] = float(double(w[e]) - double(lr) * g[e]);",
                          "w[e] = float(double(w[e]) + double(lr) * g[e]);"),
    "update_without_lr": ("w[e] = float(double(w[e]) - double(lr) * g[e]);",
                          "w[e] = float(double(w[e]) - g[e]);"),
    "update_segment_drops_last": (
        "for (int64_t i = d.seg_off[u]; i < d.seg_off[u + 1]; ++i) {\n      const float* g",
        "for (int64_t i = d.seg_off[u]; i < d.seg_off[u + 1] - 1; ++i) {\n      const float* g"),
    "update_gradient_of_wrong_bag": ("const float* g = dY + int64_t(d.sorted_bag[i]) * E;",
                                     "const float* g = dY + int64_t(d.sorted_bag[i] % B) * E;"),
    "update_last_lookup_only": ("      for (int e = 0; e < E; ++e) acc[e] += double(g[e]);",
                                "      for (int e = 0; e < E; ++e) acc[e] = double(g[e]);"),
    # validation
    "offsets_reject_empty_bags": ("if (O[k] > O[k + 1]) return kErrOffsets;",
                                  "if (O[k] >= O[k + 1]) return kErrOffsets;"),
    "offsets_skip_last_check": ("  if (O[TB] != NS) return kErrOffsets;\n", ""),
    "indices_accept_row_M": ("if (I[s] < 0 || I[s] >= m) return kErrIndexRange;",
                             "if (I[s] < 0 || I[s] > m) return kErrIndexRange;"),
    # Split-SGD-BF16 storage (Section VII)
    "split_hi_wrong_shift": ("hi[i] = uint16_t(u >> 16);", "hi[i] = uint16_t(u >> 15);"),
    "combine_swapped_halves": ("w[i] = bits_to_float((uint32_t(hi[i]) << 16) | lo[i]);",
                               "w[i] = bits_to_float((uint32_t(lo[i]) << 16) | hi[i]);"),
    "split_update_keeps_old_lo": ("      oracle_split(&w, h + e, l + e, 1);",
                                  "      { uint16_t z; oracle_split(&w, h + e, &z, 1); }"),
    "split_update_ignores_lo": ("      oracle_combine(h + e, l + e, &w, 1);",
                                "      { const uint16_t z = 0; oracle_combine(h + e, &z, &w, 1); }"),
    # BF16 activations
    "bf16_ties_away_from_zero": ("      pick = ((down >> 16) & 1u) == 0 ? down : up;",
                                 "      pick = up;"),
    "bf16_ties_toward_zero": ("    if (dd < du)\n      pick = down;", "    if (dd <= du)\n      pick = down;"),
    "bf16_widen_wrong_shift": ("out[i] = bits_to_float(uint32_t(h[i]) << 16);",
                               "out[i] = bits_to_float(uint32_t(h[i]) << 15);"),
    "bf16_act_truncates": ("  oracle_bf16_round(y.data(), Y, int64_t(y.size()));",
                           "  for (size_t i = 0; i < y.size(); ++i) Y[i] = uint16_t(float_to_bits(y[i]) >> 16);"),
    # weighted and mean pooling
    "weighted_fwd_ignores_weights": ("const double c = a ? double(a[s]) : 1.0;",
                                     "const double c = 1.0;"),
    "weighted_bwd_ignores_weights": ("      if (a) c = double(a[s]);\n", ""),
    "mean_bwd_not_divided": ("      if (mode == kPoolMean) c = 1.0 / double(O[k + 1] - O[k]);\n", ""),
    "mean_fwd_wrong_count": ("acc[e] / double(n)", "acc[e] / double(n + 1)"),
    # the literal FP32 readings (Algorithm 1; Algorithm 3 one look-up at a time)
    "literal_fwd_reversed": (
        "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n"
        "      for (int e = 0; e < E; ++e) y[e] += W[k / B][int64_t(I[s]) * E + e];",
        "    for (int64_t s = O[k + 1] - 1; s >= O[k]; --s)\n"
        "      for (int e = 0; e < E; ++e) y[e] += W[k / B][int64_t(I[s]) * E + e];"),
    "literal_fwd_fp64_accumulator": (
        "    for (int e = 0; e < E; ++e) y[e] = 0.0f;\n"
        "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n"
        "      for (int e = 0; e < E; ++e) y[e] += W[k / B][int64_t(I[s]) * E + e];",
        "    std::vector<double> a(E, 0.0);\n"
        "    for (int64_t s = O[k]; s < O[k + 1]; ++s)\n"
        "      for (int e = 0; e < E; ++e) a[e] += W[k / B][int64_t(I[s]) * E + e];\n"
        "    for (int e = 0; e < E; ++e) y[e] = float(a[e]);"),
    "literal_update_reversed": (
        "  const float alpha = -lr;\n  for (int64_t k = 0; k < int64_t(T) * B; ++k)\n"
        "    for (int64_t i = O[k]; i < O[k + 1]; ++i) {",
        "  const float alpha = -lr;\n  for (int64_t k = int64_t(T) * B - 1; k >= 0; --k)\n"
        "    for (int64_t i = O[k + 1] - 1; i >= O[k]; --i) {"),
    "literal_update_fp64_accumulator": (
        "  const float alpha = -lr;\n"
        "  for (int64_t k = 0; k < int64_t(T) * B; ++k)\n"
        "    for (int64_t i = O[k]; i < O[k + 1]; ++i) {\n"
        "      float* w = W[k / B] + int64_t(I[i]) * E;\n"
        "      for (int e = 0; e < E; ++e) {\n"
        "        const float step = alpha * dW[i * E + e];\n"
        "        w[e] = w[e] + step;\n"
        "      }\n"
        "    }",
        "  const float alpha = -lr;\n"
        "  std::vector<std::vector<double>> acc(T);\n"
        "  for (int t = 0; t < T; ++t) acc[t].assign(W[t], W[t] + rows[t] * E);\n"
        "  for (int64_t k = 0; k < int64_t(T) * B; ++k)\n"
        "    for (int64_t i = O[k]; i < O[k + 1]; ++i)\n"
        "      for (int e = 0; e < E; ++e)\n"
        "        acc[k / B][int64_t(I[i]) * E + e] += double(alpha) * dW[i * E + e];\n"
        "  for (int t = 0; t < T; ++t)\n"
        "    for (int64_t j = 0; j < rows[t] * E; ++j) W[t][j] = float(acc[t][j]);"),
}


def _build_and_check(name, old, new, tmp):
    src = open(SRC).read()
    if src.count(old) != 1:
        return name, "site", f"mutation site not found exactly once ({src.count(old)})"
    path_cpp = os.path.join(tmp, f"{name}.cpp")
    path_so = os.path.join(tmp, f"{name}.so")
    open(path_cpp, "w").write(src.replace(old, new))
    r = subprocess.run(["g++", *FLAGS, path_cpp, "-o", path_so], capture_output=True, text=True)
    if r.returncode != 0:
        return name, "build", r.stderr[-2000:]
    env = dict(os.environ, EMBBAG_ORACLE_LIB=path_so, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not slow",
                        "-p", "no:cacheprovider", os.path.join(ROOT, "tests", "test_oracle.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    failed = r.returncode != 0
    tail = "\n".join(r.stdout.strip().splitlines()[-3:])
    return name, "caught" if failed else "missed", tail


@pytest.fixture(scope="module")
def outcomes():
    with tempfile.TemporaryDirectory(prefix="oracle_mut_") as tmp:
        workers = max(1, min(8, (os.cpu_count() or 2)))
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            futs = [ex.submit(_build_and_check, n, o, w, tmp) for n, (o, w) in MUTATIONS.items()]
            res = {}
            for f in cf.as_completed(futs):
                name, verdict, info = f.result()
                res[name] = (verdict, info)
    return res


def test_unmutated_oracle_passes_its_pins():
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not slow",
                        "-p", "no:cacheprovider", os.path.join(ROOT, "tests", "test_oracle.py")],
                       cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:]


def test_harness_reports_a_harmless_edit_as_missed():
    with tempfile.TemporaryDirectory(prefix="oracle_mut_") as tmp:
        name, verdict, info = _build_and_check("noop", "constexpr int kOk = 0;",
                                               "constexpr int kOk = 0;  // unchanged", tmp)
    assert verdict == "missed", info


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(outcomes, name):
    verdict, info = outcomes[name]
    assert verdict == "caught", f"{name}: {verdict}\n{info}"
