"""Pins of proportional attention (the ln(size) key term that accompanies
size-weighted merging, Sec. III-C) at non-unit token sizes.

A token of integer size s_j stands for s_j identical tokens.  Attention in
which every key/value row j is repeated s_j times therefore gives the same
output for every query, and the probability the CLS query puts on token j
equals the summed probabilities of its copies.  That expansion is computed
here with plain (size-free) attention in float64 by library routines, so it
shares nothing with the oracle's log-bias formula.  Mutated copies of the
oracle's attention (bias on the query axis, log2 instead of ln, raw sizes
instead of their logarithm) must fail the same check.
"""
import inspect

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import fusion_oracle as fo


def _case(seed, T, H, dh, smax=6):
    rng = np.random.default_rng(seed)
    d = H * dh
    qkv = (rng.standard_normal((T, 3 * d)) * 1.5).astype(np.float32)
    s = rng.integers(1, smax + 1, size=T).astype(np.float32)
    return qkv, s


def _expanded(qkv, s, H):
    """Plain attention over keys/values repeated s_j times (float64, torch):
    output rows and the head-mean CLS probability folded back per token."""
    T, d3 = qkv.shape
    d = d3 // 3
    dh = d // H
    rep = np.repeat(np.arange(T), s.astype(np.int64))
    x = torch.from_numpy(qkv.astype(np.float64))
    q = x[:, :d].reshape(T, H, dh).transpose(0, 1)                  # [H, T, dh]
    k = x[rep, d:2 * d].reshape(len(rep), H, dh).transpose(0, 1).contiguous()
    v = x[rep, 2 * d:].reshape(len(rep), H, dh).transpose(0, 1).contiguous()
    O = F.scaled_dot_product_attention(q, k, v)                     # [H, T, dh]
    P = torch.softmax(q @ k.transpose(1, 2) / np.sqrt(dh), dim=-1)  # [H, T, Te]
    cls = np.zeros(T)
    np.add.at(cls, rep, P[:, 0, :].mean(dim=0).numpy())
    return O.transpose(0, 1).reshape(T, d).numpy(), cls


def _masked_sdpa(qkv, s, H):
    """Library attention with the additive float mask ln(s) on the key axis."""
    T, d3 = qkv.shape
    d = d3 // 3
    dh = d // H
    x = torch.from_numpy(qkv.astype(np.float64))
    q, k, v = (x[:, i * d:(i + 1) * d].reshape(T, H, dh).transpose(0, 1).contiguous()
               for i in range(3))
    mask = torch.from_numpy(np.log(s.astype(np.float64)))[None, :].expand(T, T)
    return F.scaled_dot_product_attention(q, k, v, attn_mask=mask).transpose(0, 1).reshape(T, d).numpy()


CASES = [(0, 1, 2, 8), (1, 2, 2, 8), (2, 7, 3, 16), (3, 33, 2, 16), (4, 64, 4, 8)]


def _err(attn_fn, case):
    seed, T, H, dh = case
    qkv, s = _case(seed, T, H, dh)
    O, cls = attn_fn(qkv, s, H, 1, "fp32", True)
    O_ref, cls_ref = _expanded(qkv, s, H)
    return float(np.abs(O - O_ref).max()), float(np.abs(cls - cls_ref).max())


@pytest.mark.parametrize("case", CASES)
def test_proportional_attention_equals_key_repetition(case):
    eo, ec = _err(fo.attention_heads, case)
    assert eo <= 2e-5 and ec <= 2e-6, (case, eo, ec)


@pytest.mark.parametrize("case", CASES)
def test_proportional_attention_equals_library_masked_attention(case):
    seed, T, H, dh = case
    qkv, s = _case(seed, T, H, dh)
    O, _ = fo.attention_heads(qkv, s, H, 1, "fp32", False)
    assert np.abs(O - _masked_sdpa(qkv, s, H)).max() <= 2e-5


def test_cls_attention_sums_to_one_at_any_sizes():
    for case in CASES:
        seed, T, H, dh = case
        qkv, s = _case(seed, T, H, dh)
        _, cls = fo.attention_heads(qkv, s, H, 1, "fp32", True)
        assert abs(float(cls.sum(dtype=np.float64)) - 1.0) <= 1e-5


def test_unit_sizes_make_the_term_a_no_op():
    qkv, _ = _case(7, 20, 2, 8)
    s1 = np.ones(20, dtype=np.float32)
    a = fo.attention_heads(qkv, s1, 2, 1, "fp32", True)
    b = fo.attention_heads(qkv, s1, 2, 0, "fp32", True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


MUTANTS = {
    "bias on the query axis": ("bias[None, :]", "bias[:, None]"),
    "log2 instead of ln": ("np.log(s)", "np.log2(s)"),
    "raw sizes instead of ln": ("np.log(s)", "np.asarray(s)"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutated_oracle_fails_the_pin(name):
    """A plausible mistake in the key term, planted in a copy of the oracle's
    attention, is caught by the repetition pin on at least one case."""
    old, new = MUTANTS[name]
    src = inspect.getsource(fo.attention_heads)
    assert src.count(old) == 1, "the planted mistake must replace exactly one spot"
    ns = dict(vars(fo))
    exec(compile(src.replace(old, new), "<mutant>", "exec"), ns)
    mutant = ns["attention_heads"]
    worst = max(max(_err(mutant, c)) for c in CASES)
    assert worst > 1e-3, (name, worst)
