"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake (a dropped term, a wrong sign, a transposed
operand, a wrong index, a missing step) in a copy of the numpy oracle, on the
CPU, and checks that the battery of pins (hand-derived values, closed forms,
invariants) rejects the mutant. The unmodified oracle must pass the same
battery.
"""

import json
import os
import types

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "rrq_oracle.py")

MUTATIONS = {
    "zero_point_dropped": ('q = _exact_round_sum(r, inv[:, None], z[:, None])', 'q = _exact_round_sum(r, inv[:, None], 0 * z[:, None])'),
    "zero_point_sign": ('z = np.rint((zero - lo).astype(np.float64) * inv)', 'z = np.rint((lo - zero).astype(np.float64) * inv)'),
    "range_without_zero": ("lo = np.minimum(r.min(axis=1), zero)", "lo = r.min(axis=1)"),
    "range_transposed": ("d = hi - lo ", "d = lo - hi "),
    "steps_off_by_one": ("s = d / F32(maxq)", "s = d / F32(maxq + 1)"),
    "floor_not_nearest": ('return np.rint(r.astype(np.float64) * inv.astype(np.float64) + z.astype(np.float64))', 'return np.floor(r.astype(np.float64) * inv.astype(np.float64) + z.astype(np.float64))'),
    "no_clamp": ("Q = np.clip(q, 0, maxq)", "Q = np.clip(q, -8, 8)"),
    "dequant_without_zero_point": ("qz = Q.astype(np.float32) - z[:, None]", "qz = Q.astype(np.float32)"),
    "residual_not_updated": ("r = r - rhat                           # R_k", "r = r                                  # R_k"),
    "residual_sign": ("r = r - rhat                           # R_k", "r = r + rhat                           # R_k"),
    "pack_msb_first": ("shifts = (2 * np.arange(16, dtype=np.uint32))[None, :]\n    return np.bitwise_or",
                       "shifts = (30 - 2 * np.arange(16, dtype=np.uint32))[None, :]\n    return np.bitwise_or"),
    "recon_reverse_order": ("    acc = dequant_stage(codes[0], sv(0), _stage_zeros(zeros, 0, ng, zero_point), group_size)\n    for t in range(1, k_stages):\n        acc = acc + dequant_stage(codes[t], sv(t), _stage_zeros(zeros, t, ng, zero_point),\n                                  group_size)",
                            "    last = k_stages - 1\n    acc = dequant_stage(codes[last], sv(last), _stage_zeros(zeros, last, ng, zero_point), group_size)\n    for t in range(k_stages - 2, -1, -1):\n        acc = acc + dequant_stage(codes[t], sv(t), _stage_zeros(zeros, t, ng, zero_point),\n                                  group_size)"),
    "recon_drops_last_stage": ("for t in range(1, k_stages):", "for t in range(1, k_stages - 1):"),
    "bf16_truncates": ("out = trunc + up.astype(np.uint64)", "out = trunc"),
    "degenerate_threshold_ignored": ("degenerate = s < SMALLEST_NORMAL_F32", "degenerate = s < 0"),
    "base_dequant_zero_point_sign": ("qz0 = Q0.astype(np.float32) - z0[:, None]",
                                     "qz0 = z0[:, None] - Q0.astype(np.float32)"),
    "base_zero_point_dropped": ("qz0 = Q0.astype(np.float32) - z0[:, None]",
                                "qz0 = Q0.astype(np.float32) + 0 * z0[:, None]"),
    "base_scale_dropped": ("xhat0 = qz0 * s0[:, None]", "xhat0 = qz0 * 1"),
    "base_residual_sign": ("r = x.reshape(n_groups, group_size) - xhat0",
                           "r = xhat0 - x.reshape(n_groups, group_size)"),
    "base_last_residual_stage_dropped": ("for k in range(1, n_stages):\n        Q, s, z, rhat = rtn_stage(r, bits)                  # residual stage k",
                                         "for k in range(1, n_stages - 1):\n        Q, s, z, rhat = rtn_stage(r, bits)                  # residual stage k"),
    "base_residual_not_updated": ("r = r - rhat                                         # R_k",
                                  "r = r                                                # R_k"),
    "linear_zero_point_dropped": ("return ((Q.reshape(len(rows_sel), gpr, group_size) - z[:, :, None]) * s[:, :, None]",
                                  "return ((Q.reshape(len(rows_sel), gpr, group_size) - 0 * z[:, :, None]) * s[:, :, None]"),
    "linear_scale_rows_transposed": ("s = np.asarray(s_t, dtype=np.float32).reshape(rows, gpr)[rows_sel]",
                                     "s = np.asarray(s_t, dtype=np.float32).reshape(gpr, rows).T[rows_sel]"),
    "linear_last_stage_dropped": ("    for t in range(k_stages):\n        R = stage_values_f64",
                                  "    for t in range(max(1, k_stages - 1)):\n        R = stage_values_f64"),
    "sym_zero_point_not_fixed": ("        z = np.full(lo.shape, F32(1 << (bits - 1)))",
                                 "        z = np.rint((zero - lo) * inv)"),
    "sym_range_not_widened": ("        lo, hi = zero - amax, amax", "        lo, hi = lo, hi"),
    "real_zero_point_rounded": ("        z = (zero - lo) * inv                  # fl((0 - lo) * inv)",
                                "        z = np.rint((zero - lo) * inv)"),
    "scale_not_rounded_to_storage": ("    s = round_scale(s, scale_dtype)            # the stored scale is the one used",
                                     "    s = s"),
    "zero_point_of_rounded_product": ("z = np.rint((zero - lo).astype(np.float64) * inv)",
                                      "z = np.rint(((zero - lo) * inv).astype(np.float64))"),
    "code_of_rounded_product": ("return np.rint(r.astype(np.float64) * inv.astype(np.float64) + z.astype(np.float64))",
                                "return np.rint((r * inv).astype(np.float64) + z.astype(np.float64))"),
    "pmr_single_running_sum": ("        p[j % 4] = p[j % 4] + a[:, j]", "        p[0] = p[0] + a[:, j]"),
    "pmr_sum_not_averaged": ("    mae = S / np.float32(group_size)", "    mae = S"),
    "pmr_peak_without_abs": ("    K = a.max(axis=1)", "    K = x.max(axis=1)"),
}


def _module_from(source: str) -> types.ModuleType:
    mod = types.ModuleType("rrq_oracle_mutant")
    exec(compile(source, SRC, "exec"), mod.__dict__)
    return mod


def _f(hexbits):
    return np.array([int(h, 16) for h in hexbits], dtype=np.uint32).view(np.float32)


def _battery(o) -> list:
    """Run the pins against module ``o``; return the names of failed pins."""
    failed = []
    with open(os.path.join(HERE, "golden", "hand_cases.json")) as fh:
        golden = json.load(fh)

    def check(name, fn):
        try:
            with np.errstate(all="ignore"):
                ok = fn()
        except Exception:
            ok = False
        if not ok:
            failed.append(name)

    def golden_construct():
        for case in golden["construct"]:
            x = _f(case["x"])
            bits = (x.view(np.uint32) >> 16).astype(np.uint16)
            codes, s, z = o.construct(bits, 1, x.size, case["G"], 4)
            for k, st in enumerate(case["stages"]):
                if "codes" in st and not np.array_equal(codes[k], [int(h, 16) for h in st["codes"]]):
                    return False
                if s[k].view(np.uint32)[0] != int(st["s"], 16) or z[k].view(np.uint32)[0] != int(st["z"], 16):
                    return False
            for key, want in case.get("recon_f32", {}).items():
                want_bits = x.view(np.uint32) if want == "x" else _f(want).view(np.uint32)
                if not np.array_equal(o.reconstruct(codes, s, z, case["G"], int(key)).view(np.uint32), want_bits):
                    return False
            for key, want in case.get("recon_bf16", {}).items():
                got = o.reconstruct(codes, s, z, case["G"], int(key), "bf16")
                if not np.array_equal(got, [int(h, 16) for h in want]):
                    return False
        return True

    def golden_reconstruct():
        for case in golden["reconstruct"]:
            codes = np.array([[int(h, 16) for h in row] for row in case["codes"]], dtype=np.uint32)
            sc, ze = _f(case["scales"]).reshape(-1, 1), _f(case["zeros"]).reshape(-1, 1)
            for dt, table in (("f32", case.get("recon_f32", {})), ("bf16", case.get("recon_bf16", {}))):
                for key, spec in table.items():
                    got = o.reconstruct(codes, sc, ze, case["G"], int(key), dt)
                    got = got.view(np.uint32 if dt == "f32" else np.uint16).astype(np.int64)
                    want = np.full(got.size, int(spec["default"], 16))
                    for nm, v in spec.items():
                        if nm.startswith("e"):
                            want[int(nm[1:])] = int(v, 16)
                    if not np.array_equal(got, want):
                        return False
        return True

    def invariants():
        rng = np.random.default_rng(11)
        x = (rng.standard_normal(128 * 400) * 0.02).astype(np.float32)
        x = np.where(rng.random(x.size) < 1e-2, x * 20, x).astype(np.float32)
        x = o.bf16_bits_to_f32(o.f32_to_bf16_bits(x))
        Q, s, z, rhat, _ = o.construct_f32(x, 128, 4)
        if Q.max() > 3 or not np.all(np.isin(z, [0, 1, 2, 3])):
            return False
        r = x.reshape(-1, 128)
        for k in range(4):
            r_next = (r - rhat[k].reshape(-1, 128)).astype(np.float32)
            if np.any(np.abs(r_next) > 0.5 * s[k][:, None].astype(np.float64) * (1 + 2.0 ** -20) + (s[k][:, None] == 0) * 1e30):
                return False
            r = r_next
        return True

    def crossover():
        ratios = {}
        for K in (3.0, 4.5, 6.0):
            x = np.concatenate([np.linspace(-0.5, 0.5, 127), [K]]).astype(np.float32)
            _, _, _, rhat, _ = o.construct_f32(x, 128, 2)
            rrq = (rhat[0] + rhat[1]).astype(np.float32)
            direct = o.direct_rtn_dequant(x, 128, 4)
            ratios[K] = np.abs(x - rrq.astype(np.float64)).sum() / np.abs(x - direct.astype(np.float64)).sum()
        return abs(ratios[4.5] - 1) < 1e-3 and ratios[3.0] > 1.4 and ratios[6.0] < 0.9

    def tiny_constant_degenerate():
        c = np.full(32, 2.0 ** -127, dtype=np.float32)    # bfloat16-exact, s subnormal
        bits = (c.view(np.uint32) >> 16).astype(np.uint16)
        codes, s, z = o.construct(bits, 1, 32, 32, 4)
        return np.all(s == 0) and np.all(codes == 0)

    def golden_from_base():
        with open(os.path.join(HERE, "golden", "from_base_cases.json")) as fh:
            cases = json.load(fh)["cases"]
        for case in cases:
            G, S = case["G"], case["S"]
            words = np.array([int(h, 16) for h in case["base_codes"]], dtype=np.uint32)
            s0, z0 = _f([case["base_scale"]]), _f([case["base_zero"]])
            Q0 = ((words[:, None] >> (2 * np.arange(16, dtype=np.uint32))) & 3).reshape(-1)
            xhat0 = (Q0.astype(np.float64) - float(z0[0])) * float(s0[0])
            R0 = _f(case["residual"]).astype(np.float64)[(np.arange(G) // 4) % 4]
            x = (xhat0 + R0).astype(np.float32)
            bits = (x.view(np.uint32) >> 16).astype(np.uint16)
            codes, s, z = o.construct_from_base(bits, 1, G, words, s0, z0, G, S)
            for k, st in enumerate(case["stages"]):
                if [f"{w:08X}" for w in codes[k]] != st["codes"]:
                    return False
                if f"{s[k].view(np.uint32)[0]:08X}" != st["s"] or f"{z[k].view(np.uint32)[0]:08X}" != st["z"]:
                    return False
        return True

    def from_base_identities():
        rng = np.random.default_rng(12)
        x = (rng.standard_normal(128 * 64) * 0.02).astype(np.float32)
        bits = (x.view(np.uint32) >> 16).astype(np.uint16)
        full = o.construct(bits, 1, x.size, 128, 4)
        got = o.construct_from_base(bits, 1, x.size, full[0][0], full[1][0], full[2][0], 128, 4)
        return all(np.array_equal(a, b) for a, b in zip(full, got))

    def golden_linear():
        cases = json.load(open(os.path.join(HERE, "golden", "from_base_cases.json")))["cases"]
        st = cases[0]["stages"]
        codes = np.array([[int(h, 16) for h in x["codes"]] for x in st], dtype=np.uint32)
        sc = np.stack([_f([x["s"]]) for x in st])
        ze = np.stack([_f([x["z"]]) for x in st])
        for case in json.load(open(os.path.join(HERE, "golden", "linear_cases.json")))["cases"]:
            xv = np.zeros(32, dtype=np.float32)
            if case["x"] == "ones":
                xv[:] = 1
            elif case["x"] == "alternating":
                xv[:] = np.where(np.arange(32) % 2 == 0, 1.0, -1.0)
            else:
                xv[int(case["x"].rsplit("_", 1)[1])] = 1
            xb = (xv.view(np.uint32) >> 16).astype(np.uint16).reshape(1, 32)
            for k, want in case["y"].items():
                if o.linear(codes, sc, ze, 1, 32, 32, int(k), xb)[0, 0] != want:
                    return False
        return True

    def linear_one_hot():
        rng = np.random.default_rng(13)
        rows, cols, G = 4, 128, 32
        codes = rng.integers(0, 2 ** 32, (2, rows * cols // 16), dtype=np.uint64).astype(np.uint32)
        sc = (2.0 ** rng.integers(-8, -2, (2, rows * cols // G))).astype(np.float32)
        ze = rng.integers(0, 4, (2, rows * cols // G)).astype(np.float32)
        W = o.reconstruct(codes, sc, ze, G, 2).reshape(rows, cols)
        for j in (0, 33, 127):
            xv = np.zeros(cols, dtype=np.float32)
            xv[j] = 1
            xb = (xv.view(np.uint32) >> 16).astype(np.uint16).reshape(1, cols)
            if not np.array_equal(o.linear(codes, sc, ze, rows, cols, G, 2, xb)[0], W[:, j]):
                return False
        return True

    def golden_variants():
        for case in json.load(open(os.path.join(HERE, "golden", "variant_cases.json")))["cases"]:
            x = np.full(32, case["pad"], dtype=np.float32)
            x[:len(case["x"])] = case["x"]
            bits = (x.view(np.uint32) >> 16).astype(np.uint16)
            S = 2 if "stage1" in case else 1
            _, _, _, rh = o.rtn_stage(o.bf16_bits_to_f32(bits).reshape(1, 32), 2,
                                      case["zero_point"], case["scale_dtype"])
            if [f"{int(v):08X}" for v in rh[0, :len(case["rhat0"])].view(np.uint32)] != case["rhat0"]:
                return False
            codes, sc, ze = o.construct(bits, 1, 32, 32, S, case["zero_point"], case["scale_dtype"])
            for k in range(S):
                st = case[f"stage{k}"]
                Q = ((codes[k][:, None] >> (2 * np.arange(16, dtype=np.uint32))) & 3).reshape(-1)
                want = np.full(32, st["pad_code"])
                want[:len(st["codes"])] = st["codes"]
                if not np.array_equal(Q, want):
                    return False
                got_s = (f"{int(np.asarray(sc[k]).view(np.uint16)[0]):04X}" if "s16" in st
                         else f"{int(np.asarray(sc[k]).view(np.uint32)[0]):08X}")
                if got_s != st.get("s16", st.get("s")) or f"{int(ze[k].view(np.uint32)[0]):08X}" != st["z"]:
                    return False
        return True

    def symmetric_zero_point_fixed():
        rng = np.random.default_rng(21)
        r = (rng.standard_normal((400, 32)) * 0.01).astype(np.float32)
        _, s, z, _ = o.rtn_stage(r, 2, "sym")
        return bool(np.all(z == 2.0))

    def golden_pmr():
        for case in json.load(open(os.path.join(HERE, "golden", "pmr_cases.json")))["cases"]:
            x = np.full(32, case["rest"], dtype=np.float32)
            for i, v in case["entries"]:
                x[i] = v
            if f"{int(o.group_pmr(x, 32).view(np.uint32)[0]):08X}" != case["pmr"]:
                return False
        return True

    check("golden_pmr", golden_pmr)
    check("golden_variants", golden_variants)
    check("symmetric_zero_point_fixed", symmetric_zero_point_fixed)
    check("golden_linear", golden_linear)
    check("linear_one_hot", linear_one_hot)
    check("golden_construct", golden_construct)
    check("golden_from_base", golden_from_base)
    check("from_base_identities", from_base_identities)
    check("golden_reconstruct", golden_reconstruct)
    check("invariants", invariants)
    check("crossover", crossover)
    check("tiny_constant_degenerate", tiny_constant_degenerate)
    return failed


def test_unmodified_oracle_passes_battery():
    with open(SRC) as fh:
        assert _battery(_module_from(fh.read())) == []


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutant_is_caught(name):
    with open(SRC) as fh:
        src = fh.read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, f"mutation anchor not found once: {old!r}"
    failed = _battery(_module_from(src.replace(old, new)))
    assert failed, f"mutation {name} passed every pin"
