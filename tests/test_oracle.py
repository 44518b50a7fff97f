"""The CPU oracle against its pins (closed forms, a library routine, finite
differences, gradient identities, and the paper's exact-decomposition
invariants), plus a mutation check that the pins would catch plausible
mistakes planted in the oracle."""
import json
import os
import types

import numpy as np
import pytest

import oracle
from oracle import attention as A, sp as S
from tests import oracle_pins as P
from workloads import allowed_pairs, padded_heads, workload, WORKLOADS

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.parametrize("pin", P.ATTN_PINS, ids=lambda f: f.__name__)
def test_attention_pin(pin):
    pin(A)


@pytest.mark.parametrize("pin", P.SP_PINS, ids=lambda f: f.__name__)
def test_sp_pin(pin):
    pin(S)


@pytest.mark.parametrize("pin", P.BOTH_PINS, ids=lambda f: f.__name__)
def test_decomposition_pin(pin):
    pin(A, S)


@pytest.mark.parametrize("pin", P.LOSS_PINS, ids=lambda f: f.__name__)
def test_loss_pin(pin):
    pin(oracle.loss)


def test_listing1_golden():
    """Pad count and dummy placement from Listing 1 (golden fixture)."""
    with open(os.path.join(HERE, "golden", "listing1_pad_heads.json")) as f:
        g = json.load(f)
    for c in g["cases"]:
        x = np.arange(3 * c["hs"] * 2, dtype=np.float64).reshape(1, 3, c["hs"], 2) + 1.0
        y = S.pad_heads(x, c["sp"])
        assert y.shape[2] == c["hs_new"] == padded_heads(c["hs"], c["sp"])
        zero = [h for h in range(y.shape[2]) if np.all(y[0, :, h] == 0)]
        assert zero == c["dummy_heads"]
        assert np.array_equal(S.unpad_heads(y, c["hs"]), x)


def test_dummy_heads_paper_mode():
    """Computing the zero-padded MHA dummy head (the paper's DHU) gives O = 0
    exactly and leaves real heads unchanged, so skipping it is exact."""
    rng = np.random.default_rng(11)
    L, hs, D = 10, 3, 4
    q, k, v = (rng.standard_normal((L, hs, D)) for _ in range(3))
    qp, kp, vp = (S.pad_heads(x[None], 2)[0] for x in (q, k, v))
    kw = dict(cu_q=np.array([0, L]), cu_k=np.array([0, L]), pos_q=np.arange(L), pos_k=np.arange(L),
              head_offset=0, gqa_group=1, kv_head_offset=0, scale=0.5)
    # "paper mode": treat the dummy as a real head holding zeros
    O4, _ = A.attn_forward(qp, kp, vp, H_loc=4, num_real_heads=4, **kw)
    O3, L3 = A.attn_forward(qp, kp, vp, H_loc=4, num_real_heads=3, **kw)
    assert np.all(O4[:, 3] == 0.0) and np.all(O3[:, 3] == 0.0)
    assert np.all(L3[3] == -np.inf)
    assert np.array_equal(O4[:, :3], O3[:, :3])


@pytest.mark.parametrize("name", WORKLOADS[:1] + WORKLOADS[2:3])
def test_pair_count_matches_mask(name):
    """The closed-form allowed-pair count used for FLOP accounting equals a
    brute-force count of the oracle's mask (tiny and varlen workloads)."""
    sh = workload(name)
    seg_q = A.segment_ids(sh.cu_q, sh.T_q)
    seg_k = A.segment_ids(sh.cu_k, sh.T_k)
    n = 0
    for b0 in range(0, sh.T_q, 2048):
        r = np.arange(b0, min(sh.T_q, b0 + 2048))
        n += int(A.allowed_mask(r, seg_q, seg_k, sh.pos_q, sh.pos_k, True).sum())
    assert n == allowed_pairs(sh.cu_q, sh.cu_k, sh.pos_q, sh.pos_k)


# ------------------------------------------------------------------ mutation
MUTANTS = [
    ("attention", "S = scale * (q_rows @ k.T)", "S = (q_rows @ k.T)"),
    ("attention", "m &= pos_k[None, :].astype(np.int64) <= pos_q[rows][:, None].astype(np.int64)",
     "m &= pos_k[None, :].astype(np.int64) < pos_q[rows][:, None].astype(np.int64)"),
    ("attention", "m = (sq >= 0) & (sq == seg_k[None, :])", "m = (sq >= 0) & (seg_k[None, :] >= 0)"),
    ("attention", "dS = P * (dP - Drow[:, None])", "dS = P * dP"),
    ("attention", "dk[:, kv, :] += scale * (dS.T @ q[r, h, :])", "dk[:, kv, :] += (dS.T @ q[r, h, :])"),
    ("attention", "dq[r, h, :] = scale * (dS @ k[:, kv, :])", "dq[r, h, :] = scale * (dS @ v[:, kv, :])"),
    ("attention", "dv[:, kv, :] += P.T @ dO", "dv[:, kv, :] += P.T @ do[r, h, :] * 0.5"),
    ("attention", "lse = np.where(has, m_safe + np.log(np.where(has, den, 1.0)), NEG_INF)",
     "lse = np.where(has, np.log(np.where(has, den, 1.0)), NEG_INF)"),
    ("attention", "out.append((i, g // gqa_group - kv_head_offset) if g < num_real_heads else (i, None))",
     "out.append((i, g % max(1, gqa_group) - kv_head_offset) if g < num_real_heads else (i, None))"),
    # the sampled checkers used at full size, and the bf16 decode
    ("attention", "Drow = (dO * O[:, h, :]).sum(axis=1)", "Drow = (dO * O[:, h, :])[:, :-1].sum(axis=1)"),
    ("attention", "dS = P * (dO @ v[:, kv, :].T - Drow[:, None])", "dS = P * (dO @ v[:, kv, :].T)"),
    ("attention", 'out[:, h, :] = kw["scale"] * (dS @ k[:, kv, :])', 'out[:, h, :] = (dS @ k[:, kv, :])'),
    ("attention", "need[r] = m.any(axis=1)", "need[r] = m.all(axis=1)"),
    ("attention", "m = allowed_mask(r, seg_q, seg_k[keys], pq, pk[keys], causal)",
     "m = allowed_mask(r, seg_q, seg_k[keys], pq, pk[keys] + 1, causal)"),
    ("attention", "Pk = P[:, keys]", "Pk = P[:, np.minimum(keys + 1, P.shape[1] - 1)]"),
    ("attention", "dk[:, kv, :] += kw[\"scale\"] * (dS.T @ q[r, h, :])", "dk[:, kv, :] += kw[\"scale\"] * (dS.T @ do[r, h, :])"),
    ("attention", "Drow = (dO * o_r).sum(axis=1)\n            Pk", "Drow = (dO * o_r[:, ::-1]).sum(axis=1)\n            Pk"),
    ("attention", "b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16",
     "b = (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16) | 0x8000"),
    ("attention", "return b.view(np.float32).astype(np.float64)",
     "return b.view(np.float32).astype(np.float16).astype(np.float64)"),
    ("sp", "wb = np.where(fin & np.isfinite(lb), np.exp(np.where(np.isfinite(lb), lb, 0.0) - Ls), 0.0)",
     "wb = np.where(fin & np.isfinite(lb), np.exp(np.where(np.isfinite(lb), lb, 0.0) - Ls) * 0.999, 0.0)"),
    ("sp", "pad = np.zeros(x.shape[:2] + (sp - rem,) + x.shape[3:], dtype=x.dtype)",
     "pad = np.zeros(x.shape[:2] + (sp - rem + 1,) + x.shape[3:], dtype=x.dtype)"),
    ("sp", "dst[j, :, h, :] = src[:, g, :]", "dst[j, :, h, :] = src[:, (g + 1) % src.shape[1], :]"),
    ("sp", "return np.concatenate([x, pad], axis=2)", "return np.concatenate([pad, x], axis=2)"),
    ("sp", "dst[:, g, :] += src[j, :, h, :]", "dst[:, g, :] = src[j, :, h, :]"),
    ("sp", "acc[:, g, :] = acc[:, g, :] + vals[j, :, h, :]", "acc[:, g, :] = vals[j, :, h, :]"),
    ("sp", "b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16", "b = (b + 0x8000) >> 16"),
    ("sp", "dst[:, g, :] += src[j, :, h, :]", "dst[:, g, :] += src[j, :, h, :] / max(1, sp - 1)"),
    ("sp", "                dk_g[r2][j] += a", "                dk_g[r2][j] = a"),
    ("sp", "share = [np.concatenate([r * C + np.arange(C), (n_ch - 1 - r) * C + np.arange(C)])",
     "share = [np.concatenate([r * C + np.arange(C), (n_ch - 2 - r) % n_ch * C + np.arange(C)])"),
]


def _load_mutant(module, old, new):
    srcs = {}
    for m in ("attention", "sp"):
        with open(os.path.join(os.path.dirname(oracle.__file__), m + ".py")) as f:
            srcs[m] = f.read()
    assert old in srcs[module], old
    srcs[module] = srcs[module].replace(old, new)
    pkg = types.ModuleType("oracle_mutant")
    pkg.__path__ = []
    ma = types.ModuleType("oracle_mutant.attention")
    exec(compile(srcs["attention"], "attention_mutant", "exec"), ma.__dict__)
    ms = types.ModuleType("oracle_mutant.sp")
    ms.__dict__["__package__"] = "oracle_mutant"
    import sys
    sys.modules["oracle_mutant"] = pkg
    sys.modules["oracle_mutant.attention"] = ma
    try:
        exec(compile(srcs["sp"], "sp_mutant", "exec"), ms.__dict__)
    finally:
        del sys.modules["oracle_mutant"], sys.modules["oracle_mutant.attention"]
    return ma, ms


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: f"{m[0]}:{m[2][:40]}")
def test_pins_catch_mutant(mutant):
    ma, ms = _load_mutant(*mutant)
    caught = []
    for pin in P.ATTN_PINS:
        try:
            pin(ma)
        except Exception:
            caught.append(pin.__name__)
    for pin in P.SP_PINS:
        try:
            pin(ms)
        except Exception:
            caught.append(pin.__name__)
    for pin in P.BOTH_PINS:
        try:
            pin(ma, ms)
        except Exception:
            caught.append(pin.__name__)
    assert caught, "no pin caught the planted mistake"


# plausible mistakes in the loss oracle, each caught by a loss pin
LOSS_MUTANTS = [
    ("return np.broadcast_to(u.sum(axis=0), u.shape).copy() if autograd else u.copy()",
     "return u.copy()"),
    ("    d[0::2] = -beta * sig_neg / P", "    d[0::2] = -sig_neg / P"),
    ("    return g[:, None] * (onehot - p)", "    return g[:, None] * (p - onehot)"),
    ("    g[lab == ignore_index] = 0.0", "    pass"),
    ("    lse = m + np.log(np.exp(x - m[:, None]).sum(axis=1))",
     "    lse = np.log(np.exp(x - m[:, None]).sum(axis=1))"),
    ("    loss = -scale * ps.sum()", "    loss = -scale * ps.sum() / ps.shape[0]"),
]


@pytest.mark.parametrize("mutant", LOSS_MUTANTS, ids=lambda m: m[1][:40])
def test_loss_pins_catch_mutant(mutant):
    old, new = mutant
    with open(os.path.join(os.path.dirname(oracle.__file__), "loss.py")) as f:
        src = f.read()
    assert old in src, old
    mod = types.ModuleType("loss_mutant")
    exec(compile(src.replace(old, new), "loss_mutant", "exec"), mod.__dict__)
    caught = []
    for pin in P.LOSS_PINS:
        try:
            pin(mod)
        except Exception:
            caught.append(pin.__name__)
    assert caught, "no pin caught the planted mistake"
