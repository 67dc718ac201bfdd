"""Pins for the attention-backward oracle (CPU only).

The oracle (oracle/attn_bwd_oracle.c) writes out Eq. "eq:ba" (Section 2.3):
dV = P^T dO, dP = dO V^T, dS = dsoftmax(dP), dQ = dS K, dK = dS^T Q, with the
softmax scale, GQA and the top-left causal mask, plus the row statistics
lse_i and D_i.  These tests tie it to things other than itself:
  * a library routine: torch autograd through scaled_dot_product_attention
    in float64 on the CPU (GQA by repeating K/V heads, gradients summed back);
  * brute force with a different algorithm: central finite differences of
    L = sum(O * dO) along random directions, with a numpy forward written
    here;
  * closed forms: Q = 0 (uniform softmax) gives dK = 0 and dV_j = the running
    sum of dO_i / |J_i|; lse is scipy's logsumexp of the scores; D_i equals
    <dO_i, O_i> with O from the forward oracle;
  * invariants: sum_j dK_j = 0 (softmax is blind to a common key shift),
    sum_j dV_j = sum_i dO_i (rows of P sum to one), GQA equals MHA on repeated
    K/V with the head gradients summed, future keys leave causal dQ rows
    unchanged, sampled rows equal full rows;
  * planted mistakes: copies of the C source with one plausible bug each must
    fail at least one pin.
"""

import os
import re
import shutil
import subprocess

import numpy as np
import pytest
import scipy.special
import torch

import attn_inputs as ai
import oracle


def _bits(t):
    return ai.bf16_bits(t)


def _rand(shape, seed):
    return ai.randn_bf16(shape, seed)


def _case(B, Hq, Hkv, Sq, Skv, d, seed):
    q = _rand((B, Hq, Sq, d), seed)
    k = _rand((B, Hkv, Skv, d), seed + 1)
    v = _rand((B, Hkv, Skv, d), seed + 2)
    do = _rand((B, Hq, Sq, d), seed + 3)
    return q, k, v, do


def _bwd(lib, q, k, v, do, causal, scale):
    return oracle.attn_bwd_f64(_bits(q), _bits(k), _bits(v), _bits(do), causal, scale, lib=lib)


def _autograd(q, k, v, do, causal, scale):
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    q64 = q.to(torch.float64).requires_grad_(True)
    k64 = k.to(torch.float64).requires_grad_(True)
    v64 = v.to(torch.float64).requires_grad_(True)
    o = torch.nn.functional.scaled_dot_product_attention(
        q64, k64.repeat_interleave(g, dim=1), v64.repeat_interleave(g, dim=1),
        is_causal=causal, scale=scale)
    o.backward(do.to(torch.float64))
    return q64.grad.numpy(), k64.grad.numpy(), v64.grad.numpy()


def _np_forward(q, k, v, causal, scale):
    """O in fp64 with numpy (GQA by repeating heads); a third implementation."""
    Hq, Hkv = q.shape[1], k.shape[1]
    k = np.repeat(k, Hq // Hkv, axis=1)
    v = np.repeat(v, Hq // Hkv, axis=1)
    s = scale * np.einsum("bhid,bhjd->bhij", q, k)
    if causal:
        Sq, Skv = s.shape[2], s.shape[3]
        mask = np.arange(Skv)[None, :] > np.arange(Sq)[:, None]
        s = np.where(mask, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return np.einsum("bhij,bhjd->bhid", p, v)


SHAPES = [  # B, Hq, Hkv, Sq, Skv, d, causal
    (1, 2, 2, 9, 9, 8, True),
    (2, 4, 2, 7, 11, 8, False),
    (1, 4, 1, 13, 13, 16, True),
    (1, 3, 3, 5, 12, 8, True),     # Sq < Skv, top-left causal
    (1, 2, 1, 12, 5, 8, True),     # Sq > Skv
]


def pin_autograd(lib):
    for n, (B, Hq, Hkv, Sq, Skv, d, causal) in enumerate(SHAPES):
        q, k, v, do = _case(B, Hq, Hkv, Sq, Skv, d, 100 + 10 * n)
        scale = float(np.float32(0.37))
        got = _bwd(lib, q, k, v, do, causal, scale)
        want = _autograd(q, k, v, do, causal, scale)
        for gname, a, b in zip("qkv", got, want):
            assert np.allclose(a, b, rtol=1e-9, atol=1e-11), (n, gname, np.abs(a - b).max())


def pin_finite_differences(lib):
    B, Hq, Hkv, Sq, Skv, d = 1, 2, 1, 6, 6, 4
    for causal in (False, True):
        q, k, v, do = _case(B, Hq, Hkv, Sq, Skv, d, 300 + causal)
        scale = 0.5
        dq, dk, dv = _bwd(lib, q, k, v, do, causal, scale)
        qf, kf, vf, dof = (t.to(torch.float64).numpy() for t in (q, k, v, do))
        rng = np.random.default_rng(7)
        eps = 1e-5
        for which, grad in (("q", dq), ("k", dk), ("v", dv)):
            base = {"q": qf, "k": kf, "v": vf}
            direction = rng.standard_normal(base[which].shape)

            def loss(t):
                args = dict(base)
                args[which] = base[which] + t * direction
                return float(np.sum(_np_forward(args["q"], args["k"], args["v"], causal, scale)
                                    * dof))
            fd = (loss(eps) - loss(-eps)) / (2 * eps)
            an = float(np.sum(grad * direction))
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (which, causal, fd, an)


def pin_closed_forms(lib):
    # Q = 0: P is uniform over J_i, so dK = 0 and dV_j = sum over rows that see j of dO_i/|J_i|
    B, H, S, d = 1, 2, 10, 8
    for causal in (False, True):
        _, k, v, do = _case(B, H, H, S, S, d, 400 + causal)
        q = torch.zeros((B, H, S, d), dtype=torch.bfloat16)
        dq, dk, dv = _bwd(lib, q, k, v, do, causal, 0.3)
        assert np.array_equal(dk, np.zeros_like(dk))
        dof = do.to(torch.float64).numpy()
        if causal:
            w = dof / np.arange(1, S + 1)[None, None, :, None]
            want = np.flip(np.cumsum(np.flip(w, axis=2), axis=2), axis=2)  # sum over i >= j
        else:
            want = np.broadcast_to(dof.sum(axis=2, keepdims=True) / S, dof.shape)
        assert np.allclose(dv, want, rtol=1e-12, atol=1e-12)
    # lse: scipy's logsumexp of the scores; D_i = <dO_i, O_i> with the forward oracle's O
    B, Hq, Hkv, S, d = 1, 4, 2, 9, 8
    q, k, v, do = _case(B, Hq, Hkv, S, S, d, 450)
    scale = float(np.float32(0.4))   # the oracle takes the scale as a float32
    rows = oracle.all_rows(B, Hq, S)
    lse, D = oracle.attn_row_stats_f64(_bits(q), _bits(k), _bits(v), _bits(do), rows, True,
                                       scale, lib=lib)
    qf = q.to(torch.float64).numpy()
    kf = np.repeat(k.to(torch.float64).numpy(), Hq // Hkv, axis=1)
    s = scale * np.einsum("bhid,bhjd->bhij", qf, kf)
    s = np.where(np.arange(S)[None, :] > np.arange(S)[:, None], -np.inf, s)
    assert np.allclose(lse, scipy.special.logsumexp(s, axis=-1).ravel(), rtol=1e-13, atol=1e-13)
    o = oracle.attn_fwd_f64(_bits(q), _bits(k), _bits(v), True, scale, lib=lib)
    assert np.allclose(D, np.sum(o * do.to(torch.float64).numpy(), axis=-1).ravel(),
                       rtol=1e-11, atol=1e-12)


def pin_invariants(lib):
    B, Hq, Hkv, S, d = 2, 4, 2, 11, 8
    for causal in (False, True):
        q, k, v, do = _case(B, Hq, Hkv, S, S, d, 500 + causal)
        dq, dk, dv = _bwd(lib, q, k, v, do, causal, 0.35)
        # softmax ignores a common shift of all keys of a row: sum_j dK_j = 0
        assert np.abs(dk.sum(axis=2)).max() <= 1e-12 * max(1.0, np.abs(dk).max())
        # rows of P sum to one: sum_j dV_j = sum over the group's heads and rows of dO
        dof = do.to(torch.float64).numpy().reshape(B, Hkv, Hq // Hkv, S, d)
        assert np.allclose(dv.sum(axis=2), dof.sum(axis=(2, 3)), rtol=1e-12, atol=1e-12)
        # GQA equals MHA on repeated K/V, with the gradients of a group's heads summed
        kr = k.repeat_interleave(Hq // Hkv, dim=1)
        vr = v.repeat_interleave(Hq // Hkv, dim=1)
        dq2, dk2, dv2 = _bwd(lib, q, kr, vr, do, causal, 0.35)
        assert np.allclose(dq, dq2, rtol=1e-13, atol=1e-14)
        g = Hq // Hkv
        assert np.allclose(dk, dk2.reshape(B, Hkv, g, S, d).sum(axis=2), rtol=1e-12, atol=1e-13)
        assert np.allclose(dv, dv2.reshape(B, Hkv, g, S, d).sum(axis=2), rtol=1e-12, atol=1e-13)
    # causal: keys after row i do not change dQ_i
    q, k, v, do = _case(1, 2, 2, 12, 12, 8, 520)
    dq, _, _ = _bwd(lib, q, k, v, do, True, 0.3)
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 6:] = _rand(k2[:, :, 6:].shape, 521)
    v2[:, :, 6:] = _rand(v2[:, :, 6:].shape, 522)
    dq2, _, _ = _bwd(lib, q, k2, v2, do, True, 0.3)
    assert np.array_equal(dq[:, :, :6], dq2[:, :, :6])


def pin_sampled_rows(lib):
    B, Hq, Hkv, S, d = 1, 4, 2, 10, 8
    for causal in (False, True):
        q, k, v, do = _case(B, Hq, Hkv, S, S, d, 600 + causal)
        scale = 0.3
        dq, dk, dv = _bwd(lib, q, k, v, do, causal, scale)
        rows = np.array([[0, 0, 0], [0, 3, 9], [0, 1, 4], [0, 2, 7]], np.int64)
        got = oracle.attn_bwd_dq_rows_f64(_bits(q), _bits(k), _bits(v), _bits(do), rows, causal,
                                          scale, lib=lib)
        assert np.array_equal(got, dq[rows[:, 0], rows[:, 1], rows[:, 2]])
        krows = np.array([[0, 0, 0], [0, 1, 9], [0, 1, 3], [0, 0, 6]], np.int64)
        gk, gv = oracle.attn_bwd_dkdv_rows_f64(_bits(q), _bits(k), _bits(v), _bits(do), krows,
                                               causal, scale, lib=lib)
        assert np.allclose(gk, dk[krows[:, 0], krows[:, 1], krows[:, 2]], rtol=1e-11, atol=1e-12)
        assert np.allclose(gv, dv[krows[:, 0], krows[:, 1], krows[:, 2]], rtol=1e-11, atol=1e-12)


PINS = [pin_autograd, pin_finite_differences, pin_closed_forms, pin_invariants, pin_sampled_rows]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(oracle.load())


def test_errors():
    lib = oracle.load()
    q = np.zeros((1, 3, 4, 8), np.uint16)
    k = np.zeros((1, 2, 4, 8), np.uint16)
    with pytest.raises(RuntimeError):   # Hq not a multiple of Hkv
        oracle.attn_bwd_f64(q, k, k, q, False, 1.0, lib=lib)
    with pytest.raises(RuntimeError):   # row index out of range
        oracle.attn_bwd_dq_rows_f64(q[:, :2], k, k, q[:, :2], np.array([[0, 2, 0]]), False, 1.0,
                                    lib=lib)


# ---------------------------------------------------------------- planted mistakes

MUTANTS = [
    ("no_D_subtraction", r"const double ds = prob\[j\] \* \(dp\[j\] - D\);",
     "const double ds = prob[j] * dp[j];"),
    ("dk_without_scale", r"dkh\[\(int64_t\)j \* d \+ c\] \+= P\.scale \* ds \* bf\(qi\[c\]\);",
     "dkh[(int64_t)j * d + c] += ds * bf(qi[c]);"),
    ("dk_from_keys", r"dkh\[\(int64_t\)j \* d \+ c\] \+= P\.scale \* ds \* bf\(qi\[c\]\);",
     "dkh[(int64_t)j * d + c] += P.scale * ds * bf(kj[c]);"),
    ("dv_from_ds", r"dvh\[\(int64_t\)j \* d \+ c\] \+= prob\[j\] \* bf\(doi\[c\]\);",
     "dvh[(int64_t)j * d + c] += ds * bf(doi[c]);"),
    ("gqa_strided_groups", r"for \(int hq = g \* group; hq < \(g \+ 1\) \* group; \+\+hq\) \{\n"
     r"                    for \(int i = 0; i < Sq; \+\+i\) \{\n                        double D;",
     "for (int hq = g; hq < Hq; hq += Hkv) {\n"
     "                    for (int i = 0; i < Sq; ++i) {\n                        double D;"),
    ("dp_with_keys", r"const uint16_t \*vj = kvrow\(p, p->v, b, g, j\);",
     "const uint16_t *vj = kvrow(p, p->k, b, g, j);"),
    ("causal_sees_one_more", r"return \(p->causal && i \+ 1 < p->Skv\) \? i \+ 1 : p->Skv;",
     "return (p->causal && i + 2 < p->Skv) ? i + 2 : p->Skv;"),
    ("lse_without_max", r"if \(lse\) \*lse = mx \+ log\(l\);", "if (lse) *lse = log(l);"),
]


@pytest.mark.parametrize("name,pattern,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, pattern, repl):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(os.path.join(os.path.dirname(oracle.__file__), "attn_bwd_oracle.c")).read()
    mutated, n = re.subn(pattern, repl, src)
    assert n >= 1, "mutation %s did not apply" % name
    path = tmp_path / ("m_%s.c" % name)
    path.write_text(mutated)
    so = str(tmp_path / ("m_%s.so" % name))
    try:
        oracle.build(bwd_src=str(path), out=so, extra_flags=("-Wno-unused-variable",))
    except subprocess.CalledProcessError:
        pytest.fail("mutant %s does not compile" % name)
    lib = oracle.load(so)
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(lib)
        except (AssertionError, RuntimeError):
            caught.append(pin.__name__)
    assert caught, "planted mistake %s passed every pin" % name
