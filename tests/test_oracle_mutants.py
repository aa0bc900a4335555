"""Planted mistakes in the oracle must fail its pins (no GPU).

Each case below edits a copy of oracle/orc.c in a temporary directory with
one plausible mistake (a dropped term, a wrong operand, a transposed index,
a wrong sign or rule), builds it, and runs a battery of the pins from
test_oracle_pins.py against it.  The battery must fail for every mutant and
pass for the unmodified source.  Nothing here touches the real oracle build.
"""
import json
import os

import numpy as np
import pytest

import oracle
import tracegen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "orc.c")
HAND = json.load(open(os.path.join(ROOT, "tests", "golden", "hand_examples.json")))
PIN = json.load(open(os.path.join(ROOT, "tests", "golden", "model_shapes.json")))
ADM = json.load(open(os.path.join(ROOT, "tests", "golden", "admission_examples.json")))

MUTANTS = [
    ("p feature reads c", "x[1] = S[1] * (double)p;", "x[1] = S[1] * (double)c;"),
    ("a3 term dropped", "  acc = acc + th[3] * x[3];\n", ""),
    ("a2 sign flipped", "acc = acc + th[2] * x[2];", "acc = acc - th[2] * x[2];"),
    ("a4 batch term n not n^2", "S[3] * (double)Q, (double)n * (double)n};\n    const double tm",
     "S[3] * (double)Q, (double)n};\n    const double tm"),
    ("tie goes to COMP", "const int seg = (tc > tm)", "const int seg = (tc >= tm)", 1),
    ("share uses other segment", "const double f = dot5(th[ph][seg], x);",
     "const double f = dot5(th[ph][1 - seg], x);"),
    ("phase rule and/or", "if (p[i] > 1 || c[i] == 0) prefill = 1;",
     "if (p[i] > 1 && c[i] == 0) prefill = 1;"),
    ("beta not split", "x[0] = S[0] / (double)n;", "x[0] = S[0];"),
    ("KV bytes missing K/V factor", "const int64_t s2 = 2 * L * hkv * d * kb;",
     "const int64_t s2 = L * hkv * d * kb;"),
    ("KV uses q heads", "const int64_t s2 = 2 * L * hkv * d * kb;",
     "const int64_t s2 = 2 * L * hq * d * kb;"),
    ("layer weights miss o proj", "h * d * (2 * hq + 2 * hkv)", "h * d * (hq + 2 * hkv)"),
    ("attention constant doubled", "const int64_t s3 = 2 * L * hq * d;",
     "const int64_t s3 = 4 * L * hq * d;"),
    ("coefficient index transposed", "th[ph][s][k] = (double)coeffs[(ph * 2 + s) * 5 + k];",
     "th[ph][s][k] = (double)coeffs[(s * 2 + ph) * 5 + k];"),
    ("Q sums p not p^2", "sq += (int64_t)p[i] * (int64_t)p[i];", "sq += p[i];"),
    ("output projection twice", "wb * (L * p_layer + V * h)", "wb * (L * p_layer + 2 * V * h)"),
    ("empty regime 0", "if (regime) regime[b] = ORC_REGIME_EMPTY;", "if (regime) regime[b] = 0;", 1),
    ("tenant sums of other segment", "if (tenant_sums) tenant_sums[tenant[i]] += f;",
     "if (tenant_sums) tenant_sums[tenant[i]] += dot5(th[ph][1 - seg], x);", 1),
    ("per-request p^2 uses p", "x[3] = S[3] * (double)p2;", "x[3] = S[3] * (double)p;"),
    ("admission delta sign", "if (delta) *delta = T1 - T0;", "if (delta) *delta = T0 - T1;"),
    ("admission share of the first request", "if (share) *share = f1[n];",
     "if (share) *share = f1[0];"),
    ("admission drops the candidate's context", "c1[n] = cc;", "c1[n] = 0;"),
    ("admission batch not grown", "off1[2] = {0, n + 1};", "off1[2] = {0, n > 0 ? n : 1};"),
    # the extended model (orc_attribute_ext, orc_shape_constants_ext)
    ("ext tie goes to COMP", "const int seg = (tc > tm)", "const int seg = (tc >= tm)", 2),
    ("ext empty regime 0", "if (regime) regime[b] = ORC_REGIME_EMPTY;",
     "if (regime) regime[b] = 0;", 2),
    ("ext tenant sums of other segment", "if (tenant_sums) tenant_sums[tenant[i]] += f;",
     "if (tenant_sums) tenant_sums[tenant[i]] += dot7(th[ph][1 - seg], x);", 2),
    ("ext cross term reads sum c", "S[4] * (double)R,", "S[4] * (double)C,"),
    ("ext per-request term split over the batch", "S[4] * (double)pc, S[5]};",
     "S[4] * (double)pc, S[5] / (double)n};"),
    ("ext batch term n^2", "S[5] * (double)n};", "S[5] * (double)n * (double)n};"),
    ("ext pair FLOPs halved", "const int64_t s5 = 4 * L * hq * d;",
     "const int64_t s5 = 2 * L * hq * d;"),
    ("ext logits FLOPs halved", "const int64_t s6 = 2 * V * h;", "const int64_t s6 = V * h;"),
    ("ext coefficient stride 5", "(double)coeffs[(ph * 2 + s) * 7 + k];",
     "(double)coeffs[(ph * 2 + s) * 5 + k];"),
    ("ext last term dropped", "for (int k = 1; k < 7; ++k)", "for (int k = 1; k < 6; ++k)"),
    ("ext admission: B under Eq. 1", "rc = orc_attribute_ext(1, n, off0, p, c,",
     "rc = orc_attribute(1, n, off0, p, c,"),
    ("ext admission: candidate's other-segment share", "if (share) *share = f1[n];",
     "if (share) *share = g1[n];"),
]
EXT = json.load(open(os.path.join(ROOT, "tests", "golden", "ext_examples.json")))
EXT_SETS = ("prefill_mem", "prefill_comp", "decode_mem", "decode_comp")


def ext_coeffs(sets):
    th = np.zeros(28, np.float32)
    for g, name in enumerate(EXT_SETS):
        if name in sets:
            th[g * 7:(g + 1) * 7] = sets[name]
    return th


def coeff_vec(d):
    return np.array(d["prefill_mem"] + d["prefill_comp"] + d["decode_mem"] + d["decode_comp"],
                    np.float32)


def battery(orc: oracle.Oracle):
    """A fast subset of the pins; raises AssertionError on the first miss."""
    th = coeff_vec(HAND["base_coeffs"])
    by_name = {}
    for ex in HAND["unit_shape_examples"]:
        by_name[ex["name"]] = ex
        t = th.copy()
        if ex["coeff_override"]:
            t[ex["coeff_override"]["index"]] = ex["coeff_override"]["value"]
        off = np.array([0, len(ex["p"])], np.int64)
        r = orc.attribute(off, ex["p"], ex["c"], [0] * len(ex["p"]), None, t, 1)
        assert r["T"][0] == ex["T"] and r["regime"][0] == ex["regime"]
        assert list(r["share"]) == ex["shares"]
    tt = HAND["tenant_trace"]
    tr = tracegen.from_batches([(by_name[n]["p"], by_name[n]["c"]) for n in tt["batches"]],
                               tt["tenants"], tt["n_tenants"])
    r = orc.attribute(tr.offsets, tr.p, tr.c, tr.tenant, None, th, tr.n_tenants)
    assert list(r["tenant_sums"]) == tt["tenant_sums"]
    se = HAND["shaped_examples"]
    assert list(orc.shape_constants(se["shape"])) == se["S"]
    ths = coeff_vec(se["coeffs"])
    for ex in se["examples"]:
        off = np.array([0, len(ex["p"])], np.int64)
        r = orc.attribute(off, ex["p"], ex["c"], None, se["shape"], ths, 1)
        assert r["T"][0] == ex["T"] and list(r["share"]) == ex["shares"]
    # Llama 3.1 8B published parameter count and KV bytes per token
    sh = tracegen.SHAPES["llama3.1-8b"]
    S = orc.shape_constants(sh)
    streamed = PIN["llama3_1_8b"]["total_parameters"] - sh["vocab"] * sh["hidden"] \
        - (2 * sh["n_layers"] + 1) * sh["hidden"]
    assert S[0] == 2 * streamed
    assert S[2] == PIN["llama3_1_8b"]["kv_cache_bytes_per_token_bf16"]
    # admission queries (hand-worked)
    for ex in ADM["examples"]:
        r = orc.admit(ex["p"], ex["c"], ex["cand_p"], ex["cand_c"], None, th)
        assert r["T_after"] == ex["T_after"] and r["delta"] == ex["delta"]
        assert r["regime"] == ex["regime"]
        want = ex["share"] if "share" in ex else ex["share_num"] / ex["share_den"]
        assert abs(r["share"] - want) <= 4e-16 * want
    # attention FLOPs: p^2 coefficient of the brute-force pair count
    pairs2 = 3  # (q0,k0), (q1,k0), (q1,k1)
    per_pair = sh["n_layers"] * sh["n_q_heads"] * 4 * sh["head_dim"]
    assert S[3] == (pairs2 * per_pair - 2 * 1 * per_pair) / 2
    # extended model: hand-worked batches, constants, and Eq. 1 when a5 = a6 = 0
    for ex in EXT["unit_shape_examples"]:
        off = np.array([0, len(ex["p"])], np.int64)
        r = orc.attribute(off, ex["p"], ex["c"], None, None, ext_coeffs(ex["sets"]), 0,
                          ("T", "regime", "share"), ext=True)
        assert r["T"][0] == ex["T"] and r["regime"][0] == ex["regime"]
        assert list(r["share"]) == ex["shares"]
    xs = EXT["shaped"]
    assert list(orc.shape_constants_ext(xs["shape"])) == xs["S"]
    for ex in xs["examples"]:
        off = np.array([0, len(ex["p"])], np.int64)
        r = orc.attribute(off, ex["p"], ex["c"], None, xs["shape"], ext_coeffs(xs["sets"]), 0,
                          ("T", "regime", "share"), ext=True)
        assert r["T"][0] == ex["T"] and list(r["share"]) == ex["shares"]
    Sx = orc.shape_constants_ext(sh)
    assert Sx[4] == EXT["llama3_1_8b"]["S5"] and Sx[5] == EXT["llama3_1_8b"]["S6"]
    tr = tracegen.config_trace("tiny-mixed")
    co = tracegen.config_coeffs("tiny-mixed")
    wide = np.zeros(28, np.float32)
    for g in range(4):
        wide[g * 7:g * 7 + 5] = co[g * 5:(g + 1) * 5]
    outs = ("T", "regime", "share", "tenant_sums")
    a = orc.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, co, tr.n_tenants, outs)
    b = orc.attribute(tr.offsets, tr.p, tr.c, tr.tenant, tr.shape, wide, tr.n_tenants, outs,
                      ext=True)
    for k in outs:
        assert np.array_equal(a[k], b[k]), k
    # an empty batch inside a trace: regime 255 under both models
    tr = tracegen.from_batches([([2], [0]), ([], []), ([1], [3])], None, 1)
    r = orc.attribute(tr.offsets, tr.p, tr.c, None, None, wide, 0, ("T", "regime"), ext=True)
    assert r["regime"][1] == 255 and r["T"][1] == 0.0
    # the extended admission query (hand-worked, test_oracle_admission_ext.py)
    co = np.array([8, 1, 0.5, 0, 0, 0.25, 2, 1, 2, 0, 0.25, 0, 0, 0] + [0] * 14, np.float32)
    r = orc.admit([4], [8], 2, 4, None, co, ext=True)
    assert (r["T_after"], r["delta"], r["share"], r["share_alt"], r["regime"]) == \
        (34.0, 8.0, 12.0, 5.5, 0)


def _build(tmp_path, text, tag):
    src = tmp_path / f"orc_{tag}.c"
    src.write_text(text)
    (tmp_path / "orc.h").write_text(open(os.path.join(ROOT, "oracle", "orc.h")).read())
    so = tmp_path / f"liborc_{tag}.so"
    oracle.build(str(so), str(src))
    return oracle.Oracle(str(so))


def test_battery_passes_on_real_source(tmp_path):
    battery(_build(tmp_path, open(SRC).read(), "orig"))


def mutate(text, old, new, occurrence):
    """text with the given occurrence (1-based) of old replaced; occurrence 0
    asks for a unique anchor."""
    n = text.count(old)
    if occurrence == 0:
        assert n == 1, f"mutation anchor must be unique ({n} found)"
        return text.replace(old, new)
    assert n >= occurrence, f"anchor has {n} occurrences"
    at = -1
    for _ in range(occurrence):
        at = text.index(old, at + 1)
    return text[:at] + new + text[at + len(old):]


@pytest.mark.parametrize("mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, mut):
    name, old, new = mut[:3]
    occurrence = mut[3] if len(mut) > 3 else 0
    text = open(SRC).read()
    orc = _build(tmp_path, mutate(text, old, new, occurrence), "mut")
    with pytest.raises((AssertionError, oracle.OracleError)):
        battery(orc)
