"""GPU parity of the sampling variants (specrouter_accept_and_diverge_sampled)
against the CPU reference on the same seeded inputs:

  * temperature T > 0: the tolerances of the plain rule (lengths and tokens
    bit-exact outside boundary cases, probabilities 1e-5, divergences 1e-4);
  * greedy (T = 0): every output exact -- lengths, tokens (lowest index among
    equal maxima, also across chunks), and the 0/1/+inf per-position values.
"""

import numpy as np
import pytest
import torch

import oracle
from workloads import CONFIGS, level_inputs, small_shape
from workloads.gen import bf16_bits_from_f32

from gpu_util import check_accept, run_accept

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _library():
    import paper_2505_07680_amd as sr

    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


SHAPES = [
    small_shape(name="s-f32", B=7, V=5000, gamma=(0, 6), seed=41),
    small_shape(name="s-bf16", B=6, V=12288, gamma=(1, 5), seed=42, logits="bf16"),
    small_shape(name="s-f32-wide", B=3, V=128256, gamma=(2, 4), seed=43),
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
@pytest.mark.parametrize("T", [0.5, 1.7])
def test_temperature_matches_reference(shape, T):
    inp = level_inputs(shape, kv=False)
    say(f"sampling {shape.name} T={T}")
    got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=T)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                    temperature=T)
    assert got["status"] == ref["status"] == 0
    nb, nbm = check_accept(got, ref)
    say(f"  ok ({nb} boundary, {nbm} differ)")


def _check_greedy(got, ref):
    assert got["status"] == ref["status"]
    np.testing.assert_array_equal(got["accept_len"], ref["accept_len"])
    np.testing.assert_array_equal(got["out_tokens"], ref["out_tokens"])
    for key in ("accept_prob", "p_tok", "q_tok", "tv", "kl"):
        np.testing.assert_array_equal(got[key], ref[key].astype(np.float32), err_msg=key)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
def test_greedy_matches_reference(shape):
    inp = level_inputs(shape, kv=False)
    # drafts from the draft model's argmax half of the time, so that greedy accepts happen
    from oracle.accept import decode_logits

    q = decode_logits(inp.q_logits)
    drafts = inp.drafts.copy()
    rng = np.random.default_rng(shape.seed)
    for b in range(shape.B):
        for j in range(int(inp.gamma[b])):
            if rng.random() < 0.5:
                drafts[b, j] = int(np.argmax(q[b, j]))
    say(f"greedy {shape.name}")
    got = run_accept(inp.p_logits, inp.q_logits, drafts, inp.gamma, None, None, temperature=0.0)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, drafts, inp.gamma, None, None, temperature=0.0)
    _check_greedy(got, ref)
    say(f"  ok (mean accepted {got['accept_len'].mean():.2f})")


def test_greedy_ties_resolve_to_the_lowest_index_across_chunks():
    B, G, V = 4, 3, 128256
    rng = np.random.default_rng(7)
    P = rng.normal(0, 1, (B, G + 1, V)).astype(np.float32)
    Q = rng.normal(0, 1, (B, G, V)).astype(np.float32)
    # equal maxima in different chunks, in different waves of one chunk, and in one lane
    for b, spots in enumerate([(70000, 5000), (9000, 4100), (3, 1), (128255, 64)]):
        for j in range(G + 1):
            P[b, j, list(spots)] = 50.0
        for j in range(G):
            Q[b, j, list(spots)] = 40.0
    drafts = np.tile(np.array([[5000, 4100, 1, 64]]).T, (1, G)).astype(np.int32)
    gamma = np.full(B, G, np.int32)
    got = run_accept(P, Q, drafts, gamma, None, None, temperature=0.0)
    ref = oracle.accept_and_diverge(P, Q, drafts, gamma, None, None, temperature=0.0)
    _check_greedy(got, ref)
    assert (got["accept_len"] == G).all()
    # bf16 logits tie often by themselves
    Pb, Qb = bf16_bits_from_f32(np.round(P)), bf16_bits_from_f32(np.round(Q))
    got = run_accept(Pb, Qb, drafts, gamma, None, None, temperature=0.0)
    ref = oracle.accept_and_diverge(Pb, Qb, drafts, gamma, None, None, temperature=0.0)
    _check_greedy(got, ref)


def test_config2_shaped_temperature_and_greedy_sampled():
    shape = CONFIGS[2]
    inp = level_inputs(shape, kv=False)
    seqs = [0, 5, 11, 15]
    for T in (0.8, 0.0):
        say(f"config2 T={T}")
        ua = None if T == 0 else inp.u_acc
        ur = None if T == 0 else inp.u_res
        got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, ua, ur, temperature=T)
        ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, ua, ur, seqs=seqs,
                                        temperature=T)
        if T == 0:
            for b in seqs:
                assert got["accept_len"][b] == ref["accept_len"][b]
                np.testing.assert_array_equal(got["out_tokens"][b], ref["out_tokens"][b])
                np.testing.assert_array_equal(got["tv"][b], ref["tv"][b].astype(np.float32))
        else:
            check_accept(got, ref, seqs=seqs)


# ---------------------------------------------------------------- top-k / top-p

def _check_filtered(got, ref):
    """check_accept on the sequences whose filtered sets the reference
    decides with a margin (fp32 top-p sums may differ right at p)."""
    keep = [b for b in range(ref["accept_len"].shape[0]) if not ref["filter_boundary"][b]]
    nb, nbm = check_accept(got, ref, seqs=keep)
    return len(ref["accept_len"]) - len(keep), nb, nbm


FILTERS = [(1, 1.0), (7, 1.0), (50, 1.0), (0, 0.5), (0, 0.9), (20, 0.8), (3000, 0.95)]


@pytest.mark.parametrize("shape", SHAPES[:2], ids=lambda s: s.name)
@pytest.mark.parametrize("top_k,top_p", FILTERS)
def test_top_k_top_p_match_reference(shape, top_k, top_p):
    inp = level_inputs(shape, kv=False)
    T = 0.8
    say(f"filtered {shape.name} T={T} top_k={top_k} top_p={top_p}")
    got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=T,
                     top_k=top_k, top_p=top_p)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                    temperature=T, top_k=top_k, top_p=top_p)
    assert got["status"] == ref["status"] == 0
    nf, nb, nbm = _check_filtered(got, ref)
    say(f"  ok ({nf} filter-boundary sequences skipped, {nb} boundary, {nbm} differ)")


# Enough rows for at least two threshold workgroups per CU on a 256-CU device
# (B (2 gamma_max + 1) >= 512): the threshold kernel runs its 512-thread width
# there, and its 1024-thread width on the smaller shapes above.
MANY_ROWS = [
    small_shape(name="rows-f32", B=40, V=5000, gamma=(1, 8), seed=48),
    small_shape(name="rows-bf16", B=40, V=12288, gamma=(1, 8), seed=49, logits="bf16"),
]


@pytest.mark.parametrize("shape", MANY_ROWS, ids=lambda s: s.name)
@pytest.mark.parametrize("top_k,top_p", [(1, 1.0), (50, 1.0), (0, 0.9), (20, 0.8), (3000, 0.95)])
def test_filters_with_many_rows(shape, top_k, top_p):
    inp = level_inputs(shape, kv=False)
    assert inp.B * (2 * int(np.max(inp.gamma)) + 1) >= 512
    T = 0.8
    say(f"filtered {shape.name} T={T} top_k={top_k} top_p={top_p}")
    got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=T,
                     top_k=top_k, top_p=top_p)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                    temperature=T, top_k=top_k, top_p=top_p)
    assert got["status"] == ref["status"] == 0
    nf, nb, nbm = _check_filtered(got, ref)
    say(f"  ok ({nf} filter-boundary sequences skipped, {nb} boundary, {nbm} differ)")


@pytest.mark.parametrize("logits", ["f32", "bf16"])
@pytest.mark.parametrize("top_k,top_p", [(9000, 1.0), (0, 0.5), (9000, 0.6), (40, 0.7)])
def test_filters_on_a_narrow_logit_range(logits, top_k, top_p):
    """Every logit in [1, 1.1): the whole row shares one first-level digit of
    the threshold search, more keys than its LDS candidate buffer holds, so
    the search reads the row at every level. The logits sit on a grid of 512
    values (ties of ~40 keys; bf16 rounds them to 13 values), so that top-p's
    cumulative masses move in steps well above the boundary margin."""
    shape = small_shape(name=f"narrow-{logits}", B=6, V=20000, gamma=(1, 3), seed=71, logits=logits)
    inp = level_inputs(shape, kv=False)
    rng = np.random.default_rng(71)

    def narrow(like):
        z = (1.0 + 0.1 * rng.integers(0, 512, like.shape) / 512.0).astype(np.float32)
        return (z.view(np.uint32) >> 16).astype(np.uint16) if logits == "bf16" else z

    p_l, q_l = narrow(inp.p_logits), narrow(inp.q_logits)
    say(f"narrow logits {logits} top_k={top_k} top_p={top_p}")
    got = run_accept(p_l, q_l, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=0.8, top_k=top_k,
                     top_p=top_p)
    ref = oracle.accept_and_diverge(p_l, q_l, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=0.8,
                                    top_k=top_k, top_p=top_p)
    assert got["status"] == ref["status"] == 0
    nf, nb, nbm = _check_filtered(got, ref)
    assert nf < shape.B
    say(f"  ok ({nf} filter-boundary sequences skipped, {nb} boundary, {nbm} differ)")


def test_top_k_one_with_argmax_drafts_is_greedy_on_device():
    shape = small_shape(name="k1", B=8, V=12288, gamma=(2, 6), seed=44, logits="bf16")
    inp = level_inputs(shape, kv=False)
    from oracle.accept import decode_logits

    q = decode_logits(inp.q_logits)
    drafts = inp.drafts.copy()
    for b in range(shape.B):
        for j in range(int(inp.gamma[b])):
            drafts[b, j] = int(np.argmax(q[b, j]))  # what a one-hot draft distribution emits
    got = run_accept(inp.p_logits, inp.q_logits, drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.3, top_k=1)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, drafts, inp.gamma, None, None, temperature=0.0)
    np.testing.assert_array_equal(got["accept_len"], ref["accept_len"])
    np.testing.assert_array_equal(got["out_tokens"], ref["out_tokens"])


def test_filters_off_are_the_plain_rule():
    shape = SHAPES[0]
    inp = level_inputs(shape, kv=False)
    a = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=0.8)
    for k, p in ((0, 1.0), (shape.V, 1.0), (shape.V + 7, 1.0)):
        b = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=0.8,
                       top_k=k, top_p=p)
        for key in a:
            np.testing.assert_array_equal(np.asarray(b[key]), np.asarray(a[key]), err_msg=key)


def test_filtered_config2_shape():
    """The filter at the paper-scale vocabulary (one sequence sampled per row kind)."""
    inp = level_inputs(CONFIGS[2], kv=False)
    seqs = [0, 7]
    say("filtered config 2 shape: top_k 40, top_p 0.9")
    got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.0,
                     top_k=40, top_p=0.9)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                                    temperature=1.0, top_k=40, top_p=0.9, seqs=seqs)
    assert got["status"] == 0
    keep = [b for b in seqs if not ref["filter_boundary"][b]]
    check_accept(got, ref, seqs=keep)


@pytest.mark.parametrize("logits", ["f32", "bf16"])
def test_filtered_calls_are_bitwise_deterministic(logits):
    """Top-p decides on bin masses summed by LDS atomics in whatever order the
    lanes arrive; as fixed-point integers those sums, and so every decision
    and output, must not depend on that order (Section 4.1's logits
    processors): repeated calls give identical bits."""
    shape = small_shape(name=f"det-{logits}", B=16, V=128256, gamma=(3, 6), seed=47, logits=logits)
    inp = level_inputs(shape, kv=False)
    for k, p in ((0, 0.9), (50, 0.9), (50, 1.0)):
        runs = [run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res,
                           temperature=0.7, top_k=k, top_p=p) for _ in range(3)]
        assert runs[0]["status"] == 0
        for r in runs[1:]:
            for key in runs[0]:
                np.testing.assert_array_equal(np.asarray(r[key]), np.asarray(runs[0][key]), err_msg=f"{key} k={k} p={p}")
        say(f"filtered determinism {logits} top_k {k} top_p {p}: 3 identical calls")


def _concentrate(z, dtype, n_hot, level, rng):
    """Raise n_hot entries of every row, all in the share of the filter's
    first thread (16-byte vectors 0, 1024, 2048, ... of a row whose start is
    16-byte aligned), to about `level`."""
    per_vec = 4 if dtype == "f32" else 8
    pos = np.array([1024 * per_vec * m + i for m in range(n_hot) for i in range(per_vec)])[:n_hot]
    out = z.copy()
    out[..., pos] = level + 0.05 * rng.standard_normal(out[..., pos].shape)
    return out


# (few rows: the threshold kernel's 1024-thread width; many rows, at least
# two workgroups per CU: its 512-thread width, whose thread 0 holds vectors
# 0, 512, 1024, ..., so the crowded keys still sit in one thread's share.
# Both keep gamma <= 2: with more rows per sequence nearly every sequence
# holds some row whose top-p margin is under the boundary limit, and no
# sequence would be left to compare.)
ROWS = {"few-rows": (3, (1, 2)), "many-rows": (180, (1, 2))}


@pytest.mark.parametrize("rows", list(ROWS))
@pytest.mark.parametrize("logits", ["f32", "bf16"])
@pytest.mark.parametrize("top_k,top_p,n_hot,level", [(50, 1.0, 40, 12.0), (0, 0.9, 30, 14.0), (50, 0.9, 40, 12.0)])
def test_filter_when_the_largest_keys_crowd_one_thread(rows, logits, top_k, top_p, n_hot, level):
    """Most of the kept keys sit in one thread's share of the row, more than
    the keys a thread keeps as candidates: the one-read selection cannot
    vouch for its threshold and gathers the keys above its own (lower)
    threshold in a second read; results match the reference (Section 4.1's
    logits processors)."""
    from oracle.accept import decode_logits

    V = 128256  # rows 16-byte aligned in both dtypes
    B, gam = ROWS[rows]
    shape = small_shape(name=f"crowd-{logits}-{rows}", B=B, V=V, gamma=gam, seed=73, logits=logits)
    inp = level_inputs(shape, kv=False)
    rng = np.random.default_rng(73)
    p = _concentrate(decode_logits(inp.p_logits), logits, n_hot, level, rng)
    q = _concentrate(decode_logits(inp.q_logits), logits, n_hot, level, rng)
    if logits == "bf16":
        p, q = bf16_bits_from_f32(p.astype(np.float32)), bf16_bits_from_f32(q.astype(np.float32))
    else:
        p, q = p.astype(np.float32), q.astype(np.float32)
    got = run_accept(p, q, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.0, top_k=top_k, top_p=top_p)
    ref = oracle.accept_and_diverge(p, q, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.0,
                                    top_k=top_k, top_p=top_p)
    assert got["status"] == ref["status"] == 0
    nf, nb, nbm = _check_filtered(got, ref)
    assert nf < shape.B
    say(f"crowded {logits} top_k={top_k} top_p={top_p}: ok ({nf} filter-boundary skipped)")


@pytest.mark.parametrize("rows", list(ROWS))
@pytest.mark.parametrize("logits", ["f32", "bf16"])
def test_top_p_keeping_most_of_a_flat_row(rows, logits):
    """Nearly equal logits: top-p 0.9 keeps about 90% of 20000 keys, more
    than the candidates and more than LDS holds, so the threshold comes from
    the radix select over the row itself."""
    B, gam = ROWS[rows]
    shape = small_shape(name=f"flat-{logits}-{rows}", B=B + 1, V=20000, gamma=gam, seed=74, logits=logits)
    inp = level_inputs(shape, kv=False)
    rng = np.random.default_rng(74)
    # 64 distinct values (ties of ~300 keys), so that the cumulative masses
    # move in steps well above the boundary margin
    z = lambda like: (0.05 * rng.integers(0, 64, like.shape) / 64.0).astype(np.float32)  # noqa: E731
    p, q = z(inp.p_logits), z(inp.q_logits)
    if logits == "bf16":
        p, q = bf16_bits_from_f32(p), bf16_bits_from_f32(q)
    got = run_accept(p, q, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.0, top_p=0.9)
    ref = oracle.accept_and_diverge(p, q, inp.drafts, inp.gamma, inp.u_acc, inp.u_res, temperature=1.0, top_p=0.9)
    assert got["status"] == ref["status"] == 0
    nf, nb, nbm = _check_filtered(got, ref)
    assert nf < shape.B
    say(f"flat {logits} top_p 0.9: ok ({nf} filter-boundary skipped)")
