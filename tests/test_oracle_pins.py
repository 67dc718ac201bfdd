"""Pins for the attention oracle (CPU only).

The oracle (oracle/attn_oracle.c) is the plain definition of Eq. "eq:fa"
(Section 2.3) with GQA and a top-left causal mask.  These tests tie it to
things other than itself:
  * closed forms: Q = 0 gives a uniform softmax (mean / running mean of V);
    a one-hot V reads out the probability matrix; causal row 0 is V[0];
  * a library routine: torch's scaled_dot_product_attention in float64 on the
    CPU (GQA by repeating K/V heads);
  * brute force with a different algorithm: a one-pass running-maximum
    softmax in pure Python on tiny shapes;
  * invariants: future keys do not affect causal rows, joint K/V row
    permutation, Q row permutation, (alpha*Q, scale/alpha), batch
    independence, sampled rows == full rows, large scores stay finite;
  * planted mistakes: copies of the C source with one plausible bug each
    (wrong GQA head, off-by-one causal edge, dropped scale, transposed K,
    wrong V row, missing normalisation, no max subtraction) must fail at least
    one pin.

Every pin is a function of the loaded library so that the mutation test can
run the same pins against the planted-mistake builds.
"""

import math
import os
import re
import shutil
import subprocess

import numpy as np
import pytest
import torch

import attn_inputs as ai
import oracle

# ---------------------------------------------------------------- helpers


def _bits(t):
    return ai.bf16_bits(t)


def _f64(t):
    return t.to(torch.float64)


def _run(lib, q, k, v, causal, scale):
    return oracle.attn_fwd_f64(_bits(q), _bits(k), _bits(v), causal, scale, lib=lib)


def _rand(shape, seed):
    return ai.randn_bf16(shape, seed)


def _sdpa_f64(q, k, v, causal, scale):
    """torch SDPA in float64 on the CPU; GQA via repeat_interleave of K/V heads."""
    Hq, Hkv = q.shape[1], k.shape[1]
    kk = _f64(k).repeat_interleave(Hq // Hkv, dim=1)
    vv = _f64(v).repeat_interleave(Hq // Hkv, dim=1)
    return torch.nn.functional.scaled_dot_product_attention(
        _f64(q), kk, vv, is_causal=bool(causal), scale=float(scale)).numpy()


# ---------------------------------------------------------------- pins


def pin_zero_q_uniform(lib):
    """Q = 0: every score is 0, softmax is uniform over the visible keys."""
    B, Hq, Hkv, S, d = 2, 4, 2, 37, 16
    q = torch.zeros(B, Hq, S, d, dtype=torch.bfloat16)
    k = _rand((B, Hkv, S, d), 11)
    v = _rand((B, Hkv, S, d), 12)
    vv = _f64(v).numpy().repeat(Hq // Hkv, axis=1)
    o = _run(lib, q, k, v, False, 0.25)
    want = np.broadcast_to(vv.mean(axis=2, keepdims=True), o.shape)
    np.testing.assert_allclose(o, want, rtol=0, atol=1e-13)
    oc = _run(lib, q, k, v, True, 0.25)
    cum = np.cumsum(vv, axis=2) / np.arange(1, S + 1, dtype=np.float64)[None, None, :, None]
    np.testing.assert_allclose(oc, cum, rtol=0, atol=1e-13)


def pin_one_hot_v(lib):
    """V[j] = e_j with Skv <= d: O[i, :Skv] is row i of P, zero beyond."""
    B, H, Sq, Skv, d = 1, 2, 9, 7, 8
    q = _rand((B, H, Sq, d), 21)
    k = _rand((B, H, Skv, d), 22)
    eye = torch.zeros(B, H, Skv, d, dtype=torch.bfloat16)
    for j in range(Skv):
        eye[:, :, j, j] = 1.0
    scale = 0.5
    for causal in (False, True):
        o = _run(lib, q, k, eye, causal, scale)
        assert np.all(o[..., Skv:] == 0.0)
        np.testing.assert_allclose(o[..., :Skv].sum(-1), 1.0, rtol=0, atol=1e-14)
        s = scale * np.einsum("bhid,bhjd->bhij", _f64(q).numpy(), _f64(k).numpy())
        if causal:
            s = np.where(np.arange(Skv)[None, :] <= np.arange(Sq)[:, None], s, -np.inf)
        p = np.exp(s - s.max(-1, keepdims=True))
        p /= p.sum(-1, keepdims=True)
        np.testing.assert_allclose(o[..., :Skv], p, rtol=0, atol=1e-14)
    # Q = 0 as well: O[i, j] = 1/|J_i| for the visible j
    o = _run(lib, torch.zeros_like(q), k, eye, True, scale)
    for i in range(Sq):
        n = min(i + 1, Skv)
        np.testing.assert_allclose(o[0, 0, i, :n], 1.0 / n, rtol=0, atol=1e-15)
        assert np.all(o[0, 0, i, n:] == 0.0)


def pin_causal_first_row(lib):
    """Causal row 0 sees key 0 only: O[0] == V[0] exactly."""
    B, Hq, Hkv, S, d = 2, 6, 3, 20, 32
    q, k, v = (_rand((B, Hq, S, d), 31), _rand((B, Hkv, S, d), 32), _rand((B, Hkv, S, d), 33))
    o = _run(lib, q, k, v, True, 1.0 / math.sqrt(d))
    vv = _f64(v).numpy().repeat(Hq // Hkv, axis=1)
    assert np.array_equal(o[:, :, 0, :], vv[:, :, 0, :])


def pin_library_sdpa(lib):
    """Agreement with torch SDPA (float64, CPU) on ragged, GQA and causal shapes."""
    cases = [(1, 1, 1, 1, 1, 8, False), (2, 4, 2, 13, 13, 16, True), (1, 8, 1, 5, 29, 32, False),
             (1, 8, 2, 29, 29, 64, True), (3, 2, 2, 33, 17, 8, False), (1, 4, 4, 40, 40, 128, True)]
    for n, (B, Hq, Hkv, Sq, Skv, d, causal) in enumerate(cases):
        q = _rand((B, Hq, Sq, d), 100 + 3 * n)
        k = _rand((B, Hkv, Skv, d), 101 + 3 * n)
        v = _rand((B, Hkv, Skv, d), 102 + 3 * n)
        scale = ai.default_scale(d)
        o = _run(lib, q, k, v, causal, scale)
        np.testing.assert_allclose(o, _sdpa_f64(q, k, v, causal, scale), rtol=0, atol=1e-12)


def _one_pass_row(qrow, K, V, scale, jend):
    """Running-maximum (online) softmax over keys 0..jend-1, pure Python."""
    m, l = -math.inf, 0.0
    acc = [0.0] * len(V[0])
    for j in range(jend):
        s = scale * sum(a * b for a, b in zip(qrow, K[j]))
        m_new = max(m, s)
        alpha = math.exp(m - m_new) if m != -math.inf else 0.0
        p = math.exp(s - m_new)
        l = l * alpha + p
        acc = [a * alpha + p * x for a, x in zip(acc, V[j])]
        m = m_new
    return [a / l for a in acc]


def pin_brute_force_tiny(lib):
    """A different algorithm (one-pass online softmax) on tiny shapes."""
    for n, (B, Hq, Hkv, Sq, Skv, d, causal) in enumerate(
            [(2, 4, 2, 8, 8, 8, True), (1, 2, 1, 5, 7, 4, False), (2, 3, 3, 6, 3, 2, True)]):
        q = _rand((B, Hq, Sq, d), 200 + 3 * n)
        k = _rand((B, Hkv, Skv, d), 201 + 3 * n)
        v = _rand((B, Hkv, Skv, d), 202 + 3 * n)
        scale = float(np.float32(0.7))  # the float32 value the oracle receives
        o = _run(lib, q, k, v, causal, scale)
        Q, K, V = (_f64(t).tolist() for t in (q, k, v))
        for b in range(B):
            for h in range(Hq):
                g = h // (Hq // Hkv)
                for i in range(Sq):
                    jend = min(i + 1, Skv) if causal else Skv
                    want = _one_pass_row(Q[b][h][i], K[b][g], V[b][g], scale, jend)
                    np.testing.assert_allclose(o[b, h, i], want, rtol=0, atol=1e-12)


def pin_gqa_is_repeated_mha(lib):
    """GQA with Hkv heads equals MHA on K/V heads repeated Hq/Hkv times (contiguous groups)."""
    B, Hq, Hkv, S, d = 2, 8, 2, 19, 16
    q, k, v = (_rand((B, Hq, S, d), 41), _rand((B, Hkv, S, d), 42), _rand((B, Hkv, S, d), 43))
    for causal in (False, True):
        o = _run(lib, q, k, v, causal, 0.3)
        o2 = _run(lib, q, k.repeat_interleave(Hq // Hkv, dim=1),
                  v.repeat_interleave(Hq // Hkv, dim=1), causal, 0.3)
        assert np.array_equal(o, o2)


def pin_invariants(lib):
    B, H, S, d = 2, 3, 24, 16
    q, k, v = (_rand((B, H, S, d), 51), _rand((B, H, S, d), 52), _rand((B, H, S, d), 53))
    scale = 0.25
    # causal: rows i are unaffected by keys/values j > i
    oc = _run(lib, q, k, v, True, scale)
    k2, v2 = k.clone(), v.clone()
    k2[:, :, 12:] = _rand((B, H, S - 12, d), 54)
    v2[:, :, 12:] = _rand((B, H, S - 12, d), 55)
    oc2 = _run(lib, q, k2, v2, True, scale)
    assert np.array_equal(oc[:, :, :12], oc2[:, :, :12])
    assert not np.allclose(oc[:, :, 12:], oc2[:, :, 12:])
    # non-causal: joint permutation of K/V rows leaves O unchanged
    o = _run(lib, q, k, v, False, scale)
    perm = torch.randperm(S, generator=torch.Generator().manual_seed(5))
    o_p = _run(lib, q, k[:, :, perm], v[:, :, perm], False, scale)
    np.testing.assert_allclose(o, o_p, rtol=0, atol=1e-13)
    # permuting Q rows permutes O rows
    o_q = _run(lib, q[:, :, perm], k, v, False, scale)
    assert np.array_equal(o_q, o[:, :, perm.numpy()])
    # (alpha Q, scale/alpha) with alpha a power of two is the same problem exactly
    o_a = _run(lib, q * 4, k, v, False, scale / 4)
    assert np.array_equal(o_a, o)
    # batches are independent
    o_b1 = _run(lib, q[1:], k[1:], v[1:], False, scale)
    assert np.array_equal(o_b1, o[1:])


def pin_rows_match_full(lib):
    B, Hq, Hkv, Sq, Skv, d = 2, 4, 2, 33, 45, 32
    q, k, v = (_rand((B, Hq, Sq, d), 61), _rand((B, Hkv, Skv, d), 62), _rand((B, Hkv, Skv, d), 63))
    rows = ai.sample_rows(B, Hq, Sq, 16, 5, seed=7)
    for causal in (False, True):
        full = _run(lib, q, k, v, causal, 0.2)
        part = oracle.attn_fwd_rows_f64(_bits(q), _bits(k), _bits(v), rows, causal, 0.2, lib=lib)
        assert np.array_equal(part, full[rows[:, 0], rows[:, 1], rows[:, 2]])


def pin_large_scores_finite(lib):
    """Scores around +-1e3: the max subtraction keeps exp() finite."""
    B, H, S, d = 1, 2, 16, 16
    q = _rand((B, H, S, d), 71) * 64
    k = _rand((B, H, S, d), 72) * 64
    v = _rand((B, H, S, d), 73)
    for causal in (False, True):
        o = _run(lib, q, k, v, causal, 0.25)
        assert np.all(np.isfinite(o))
        np.testing.assert_allclose(o, _sdpa_f64(q, k, v, causal, 0.25), rtol=0, atol=1e-12)


PINS = [pin_zero_q_uniform, pin_one_hot_v, pin_causal_first_row, pin_library_sdpa,
        pin_brute_force_tiny, pin_gqa_is_repeated_mha, pin_invariants, pin_rows_match_full,
        pin_large_scores_finite]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(oracle.load())


def test_errors():
    lib = oracle.load()
    q = np.zeros((1, 3, 4, 8), np.uint16)
    k = np.zeros((1, 2, 4, 8), np.uint16)
    with pytest.raises(RuntimeError):   # Hq not a multiple of Hkv
        oracle.attn_fwd_f64(q, k, k, False, 1.0, lib=lib)
    rows = np.array([[0, 0, 4]], np.int64)  # row index out of range
    with pytest.raises(RuntimeError):
        oracle.attn_fwd_rows_f64(q[:, :2], k, k, rows, False, 1.0, lib=lib)


# ---------------------------------------------------------------- planted mistakes

# (name, regex on the oracle source, replacement); each is a plausible bug.
MUTANTS = [
    ("gqa_head_modulo", r"const int g = hq / group;", "const int g = hq % Hkv;"),
    ("causal_off_by_one", r"jend = i \+ 1;", "jend = i + 2 < Skv ? i + 2 : Skv;"),
    ("scale_dropped", r"s\[j\] = scale \* dot;", "s[j] = dot;"),
    ("k_transposed", r"bf16_bits_to_double\(krow\[c\]\)",
     "bf16_bits_to_double(kh[(int64_t)c * Skv + j])"),
    ("v_row_reversed", r"const uint16_t \*vrow = vh \+ \(int64_t\)j \* d;",
     "const uint16_t *vrow = vh + (int64_t)(jend - 1 - j) * d;"),
    ("no_normalisation", r"for \(int c = 0; c < d; \+\+c\) out\[c\] /= l;", ""),
    ("no_max_subtraction", r"exp\(s\[j\] - mx\)", "exp(s[j])"),
    ("max_over_all_keys", r"for \(int j = 0; j < jend; \+\+j\)\n        if \(s\[j\] > mx\)",
     "for (int j = 0; j < Skv && j < jend + 1; ++j)\n        if (s[j] > mx)"),
]


@pytest.mark.parametrize("name,pattern,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, pattern, repl):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = open(os.path.join(os.path.dirname(oracle.__file__), "attn_oracle.c")).read()
    mutated, n = re.subn(pattern, repl, src)
    assert n >= 1, "mutation %s did not apply" % name
    path = tmp_path / ("m_%s.c" % name)
    path.write_text(mutated)
    so = str(tmp_path / ("m_%s.so" % name))
    try:
        oracle.build(src=str(path), out=so, extra_flags=("-Wno-unused-variable",))
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


def test_oracle_c_under_address_and_ub_sanitizers(tmp_path):
    """The C oracle (forward, sampled rows, row statistics, backward) on ragged
    GQA shapes, built for the host with AddressSanitizer and UBSan: no
    out-of-bounds access, leak or undefined behaviour, and finite results."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not installed")
    here = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")
    drv = tmp_path / "drv.c"
    drv.write_text(r'''
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
int oracle_attn_fwd_f64(const uint16_t*, const uint16_t*, const uint16_t*, double*, int, int, int,
                        int, int, int, int, float, int);
int oracle_attn_fwd_rows_f64(const uint16_t*, const uint16_t*, const uint16_t*, const int64_t*,
                             int64_t, double*, int, int, int, int, int, int, int, float, int);
int oracle_attn_bwd_f64(const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*,
                        double*, double*, double*, int, int, int, int, int, int, int, float, int);
int oracle_attn_row_stats_f64(const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*,
                              const int64_t*, int64_t, double*, double*, int, int, int, int, int,
                              int, int, float, int);
static uint16_t *rnd(size_t n, unsigned s) {
    uint16_t *p = malloc(n * sizeof *p);
    for (size_t i = 0; i < n; ++i) { s = s * 1103515245u + 12345u; p[i] = 0x3c00 | (s >> 16 & 0x7f) | ((s >> 8) & 0x8000); }
    return p;
}
static int finite(const double *x, size_t n) { for (size_t i = 0; i < n; ++i) if (!isfinite(x[i])) return 0; return 1; }
int main(void) {
    const int shapes[][7] = {{2, 4, 2, 5, 7, 8, 1}, {1, 3, 1, 9, 4, 16, 0}, {1, 2, 2, 1, 1, 8, 1}};
    for (int c = 0; c < 3; ++c) {
        const int B = shapes[c][0], Hq = shapes[c][1], Hkv = shapes[c][2], Sq = shapes[c][3];
        const int Skv = shapes[c][4], d = shapes[c][5], causal = shapes[c][6];
        const size_t nq = (size_t)B * Hq * Sq * d, nk = (size_t)B * Hkv * Skv * d;
        uint16_t *q = rnd(nq, 1 + c), *k = rnd(nk, 2 + c), *v = rnd(nk, 3 + c), *dout = rnd(nq, 4 + c);
        double *o = malloc(nq * sizeof *o), *dq = malloc(nq * sizeof *dq);
        double *dk = malloc(nk * sizeof *dk), *dv = malloc(nk * sizeof *dv);
        const int64_t nrows = (int64_t)B * Hq * Sq;
        int64_t *rows = malloc((size_t)nrows * 3 * sizeof *rows);
        for (int64_t r = 0; r < nrows; ++r) {
            rows[3 * r] = r / ((int64_t)Hq * Sq); rows[3 * r + 1] = (r / Sq) % Hq; rows[3 * r + 2] = r % Sq;
        }
        double *orow = malloc((size_t)nrows * d * sizeof *orow), *lse = malloc((size_t)nrows * sizeof *lse);
        double *dsum = malloc((size_t)nrows * sizeof *dsum);
        const float sc = 0.35f;
        if (oracle_attn_fwd_f64(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, sc, 1)) return 10 + c;
        if (oracle_attn_fwd_rows_f64(q, k, v, rows, nrows, orow, B, Hq, Hkv, Sq, Skv, d, causal, sc, 1)) return 20 + c;
        if (oracle_attn_row_stats_f64(q, k, v, dout, rows, nrows, lse, dsum, B, Hq, Hkv, Sq, Skv, d, causal, sc, 1)) return 30 + c;
        if (oracle_attn_bwd_f64(q, k, v, dout, dq, dk, dv, B, Hq, Hkv, Sq, Skv, d, causal, sc, 1)) return 40 + c;
        for (size_t i = 0; i < nq; ++i) if (fabs(o[i] - orow[i]) > 1e-12) return 50 + c;
        if (!finite(o, nq) || !finite(lse, nrows) || !finite(dsum, nrows) || !finite(dq, nq) ||
            !finite(dk, nk) || !finite(dv, nk)) return 60 + c;
        free(q); free(k); free(v); free(dout); free(o); free(dq); free(dk); free(dv);
        free(rows); free(orow); free(lse); free(dsum);
    }
    puts("ok");
    return 0;
}
''')
    exe = tmp_path / "drv"
    cmd = [gcc, "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-Wno-unknown-pragmas", str(drv),
           os.path.join(here, "attn_oracle.c"), os.path.join(here, "attn_bwd_oracle.c"),
           "-o", str(exe), "-lm"]
    b = subprocess.run(cmd, capture_output=True, text=True)
    if b.returncode != 0 and "asan" in b.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + b.stderr[-200:])
    assert b.returncode == 0, b.stderr[-2000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr[-2000:])
