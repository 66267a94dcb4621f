"""Parity of the HIP path with the CPU oracle, through the C ABI.

Decisions (accepted_len, next_token) must match bit for bit except where the
oracle places a uniform within 1e-6 of its threshold (counted and reported);
probabilities must match within 1e-5 relative (fp32 logits) or 2e-3
(fp16 / bf16 logits)."""
import math

import numpy as np
import scipy.special
import scipy.stats
import pytest
import torch

import oracle
from paper_2406_11016_amd import binding
from paper_2406_11016_amd import workloads as W
from tests.golden_util import example_arrays
from tests.gpu_util import compare, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    binding.load_library()
    torch.cuda.init()


def _report(label, x, nflag):
    print(f"[parity] {label}: B={x.batch} gamma={x.gamma} V={x.vocab} {x.dtype} {x.mode} flagged={nflag}",
          flush=True)


# --- reduced versions of every named workload: several tiles, ragged tails --

SMALL = [
    ("exact_b1_g5_v51865_f32", dict(vocab=9001)),
    ("exact_b1_g10_v32000_f16", dict(vocab=6007)),
    ("exact_b16_g5_v51865_f32", dict(vocab=5003)),
    ("exact_b64_g8_v128256_bf16", dict(batch=8, vocab=20011)),
    ("sigmoid_b32_g10_v50272_f16_t0.7", dict(batch=8, vocab=10007)),
]


@pytest.mark.parametrize("name,over", SMALL, ids=[s[0] for s in SMALL])
def test_small_workloads(name, over):
    w = W.WORKLOADS[name].with_(**over)
    x = W.generate(w)
    nflag = compare(x, run_gpu(x), run_oracle(x), label=name)
    _report(name + " (reduced)", x, nflag)


# --- the named workloads at full size (the shapes the benchmark times) ------

@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_full_size_workloads(name):
    x = W.generate(W.WORKLOADS[name])
    nflag = compare(x, run_gpu(x), run_oracle(x), label=name)
    _report(name, x, nflag)


# --- edge cases ---------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("V", [1, 2, 7, 8, 63, 64, 65, 255, 256, 257, 4097, 8193])
def test_vocab_edge_sizes(dtype, V):
    for gamma, B in [(1, 1), (3, 5)]:
        x = W.small_case(B, gamma, V, dtype, seed=100 + V)
        compare(x, run_gpu(x), run_oracle(x), label=f"V={V} {dtype} g={gamma}")


@pytest.mark.parametrize("gamma", [1, 2, 4, 5, 6, 10, 11, 13, 16, 17, 20, 21, 31, 33, 40, 64, 65, 80, 81, 100, 128])
def test_gamma_range(gamma):
    # the row-normaliser merge groups 16, 8, 4, 2 or 1 lanes per row by the
    # number of rows (2 gamma); low noise so that long accepted prefixes occur
    for dtype, V, mode in (("f32", 3001, "exact"), ("bf16", 20011, "exact"), ("f16", 5003, "sigmoid")):
        x = W.small_case(3, gamma, V, dtype, mode=mode, seed=200 + gamma, noise_scale=0.05,
                         alpha=-1e3, beta=1e3)
        nflag = compare(x, run_gpu(x), run_oracle(x), label=f"gamma={gamma} {dtype} {mode}")
        _report(f"gamma={gamma}", x, nflag)


@pytest.mark.parametrize("B,gamma,V,dtype", [(2, 3, 65537, "f16"), (8, 8, 20011, "bf16"), (16, 2, 40000, "f32"),
                                              (16, 4, 40000, "f32")])
def test_short_stream_block_depths(B, gamma, V, dtype):
    # short streams whose stats chunks hold 1, 2, 4 and 8 vectors per lane
    # (the stats blocks take that depth); mixed acceptance, so the residual
    # and the bonus draws both run
    for noise in (0.2, 1.0):
        x = W.small_case(B, gamma, V, dtype, seed=300 + B + gamma, noise_scale=noise)
        nflag = compare(x, run_gpu(x), run_oracle(x), label=f"depths B={B} g={gamma} V={V} {dtype} noise={noise}")
        _report(f"block depths noise={noise}", x, nflag)


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_unaligned_rows_and_offsets(mode):
    # odd V in fp32: every row after the first starts off a 16-byte boundary;
    # odd V in 16-bit storage: rows start off a 4-byte boundary (element loads)
    for dt, V in (("f32", 12347), ("bf16", 12347), ("f16", 2049)):
        x = W.small_case(7, 4, V, dt, mode=mode, seed=3, alpha=-1e3, beta=1e3)
        compare(x, run_gpu(x), run_oracle(x), label=f"odd V {dt}")


@pytest.mark.parametrize("T", [0.7, 1.0, 1.3])
@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_temperatures(T, mode):
    x = W.small_case(6, 5, 3001, "f16", mode=mode, seed=11, temperature=T, alpha=-1e3, beta=1e3)
    compare(x, run_gpu(x), run_oracle(x), label=f"T={T} {mode}")


def test_identical_rows_accept_every_draft_bit_exactly():
    x = W.small_case(16, 6, 20000, "f32", seed=5)
    x.draft[:] = x.target[:, :6]
    x.uniforms[:, :6] = W.UNIFORM_MAX          # the largest uniform still accepts tau = 1
    for mode in ("exact", "sigmoid"):
        x.mode = mode
        g = run_gpu(x)
        assert np.all(g.accepted_len == 6), (mode, g.accepted_len)
        assert np.all(g.tau == 1.0), mode
        compare(x, g, run_oracle(x), label=f"p==q {mode}")


def test_token_extremes_and_uniform_extremes():
    x = W.small_case(8, 4, 777, "bf16", seed=9)
    x.tokens[0, :] = 0
    x.tokens[1, :] = 776
    x.uniforms[2, :] = 0.0
    x.uniforms[3, :] = W.UNIFORM_MAX
    x.uniforms[4, -1] = 0.0
    x.uniforms[5, -1] = W.UNIFORM_MAX
    compare(x, run_gpu(x), run_oracle(x), label="extremes")


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_masked_logits(mode):
    x = W.small_case(12, 4, 3000, "f32", mode=mode, seed=21, alpha=-1e3, beta=1e3)
    rng = np.random.default_rng(0)
    mask_t = rng.random(x.target.shape) < 0.5
    mask_d = rng.random(x.draft.shape) < 0.5
    x.target[mask_t] = -np.inf
    x.draft[mask_d] = -np.inf
    # keep some drafted tokens on target-masked positions (reject) and some on
    # draft-masked positions (tau = 1)
    compare(x, run_gpu(x), run_oracle(x), label=f"masked {mode}")


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
@pytest.mark.parametrize("k", [1, 3, 50, 2000])
def test_top_k_masked_logits(mode, k):
    # a top-k logit processor on both models: most logits -inf, different
    # supports for draft and target (tokens outside the target's top-k are
    # rejected, tokens inside are accepted with tau ~ 1 in sigmoid mode)
    for dtype, V in (("f32", 5003), ("bf16", 20011)):
        x = W.small_case(8, 6, V, dtype, mode=mode, seed=400 + k, top_k=k, alpha=-1e4, beta=1e4)
        nflag = compare(x, run_gpu(x), run_oracle(x), label=f"top-{k} {dtype} {mode}")
        _report(f"top-{k}", x, nflag)


def test_fp16_extremes():
    x = W.small_case(4, 3, 1000, "f16", seed=31)
    x.target[0, 0, 10] = np.float16(65504.0)
    x.draft[1, 0, 20] = np.float16(-65504.0)
    x.target[2, :, :] = np.float16(65504.0)
    x.draft[3, :, :] = np.float16(-65504.0)
    compare(x, run_gpu(x), run_oracle(x), label="fp16 extremes")


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_sentinels(mode):
    x = W.small_case(6, 3, 500, "f32", mode=mode, seed=41, alpha=-1e3, beta=1e3)
    x.tokens[0, 1] = 500                      # invalid token
    x.tokens[1, 0] = -3
    x.target[2, 0, :] = np.nan                # NaN in a row read by both modes
    x.uniforms[3, :] = 0.0                    # accept everything -> bonus row read
    x.target[3, 3, :] = np.nan
    x.draft[4, 2, 7] = np.nan                 # NaN away from the token: exact reads it, sigmoid does not
    x.tokens[4, 2] = 8
    x.uniforms[4, :3] = 0.0
    if mode == "exact":
        x.target[5, :2, :] = -np.inf          # all -inf rows (exact: unreadable)
    g = run_gpu(x)
    o = run_oracle(x)
    assert g.accepted_len.tolist() == o.accepted_len.tolist(), (g.accepted_len, o.accepted_len)
    assert g.next_token.tolist() == o.next_token.tolist(), (g.next_token, o.next_token)
    assert g.accepted_len[0] == -1 and g.accepted_len[1] == -1 and g.accepted_len[2] == -1
    assert g.accepted_len[3] == -1


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_bad_bonus_row_leaves_a_rejecting_element_alone(mode):
    """Target row gamma is read for the bonus draw before the decision is
    known (in both modes); a NaN there must not touch an element that rejects
    a draft, whose step never reads that row.  The first drafted token gets a
    -inf target logit, so tau = 0 and it is rejected in both modes."""
    x = W.small_case(4, 3, 700, "f32", mode=mode, seed=43, alpha=-1e3, beta=1e3)
    for b in range(4):
        x.target[b, 3, :] = np.nan
        x.target[b, 0, x.tokens[b, 0]] = -np.inf
    g = run_gpu(x)
    o = run_oracle(x)
    assert np.all(o.accepted_len == 0), o.accepted_len
    assert g.accepted_len.tolist() == o.accepted_len.tolist(), (g.accepted_len, o.accepted_len)
    compare(x, g, o, label=f"bad bonus row, rejecting {mode}")


def test_bonus_draw_with_vanishing_leading_mass():
    """Every draft accepted and the last uniform 0: the draw takes the first
    token of positive probability.  The first 50 logits of target row gamma
    are so small (p ~ e^-205) that their fp32 weights underflow even against
    the sub-chunk's own scale; the oracle (fp64) returns token 0, on a CDF
    edge, so it flags the case.  The GPU must still return a valid token: 0
    or the first token of representable weight, 50."""
    x = W.small_case(4, 3, 40000, "f32", seed=91)
    x.draft[:] = x.target[:, :3]
    x.uniforms[:, :3] = 0.0
    x.uniforms[:, 3] = 0.0
    x.target[:, 3, :50] = -200.0
    g = run_gpu(x)
    o = run_oracle(x)
    assert np.all(g.accepted_len == 3), g.accepted_len
    assert np.all((g.next_token == 0) | (g.next_token == 50)), g.next_token
    assert np.all(o.next_token == 0) and np.all(o.flagged())
    compare(x, g, o, label="vanishing leading mass")


@pytest.mark.parametrize("dtype,V", [("f32", 300007), ("bf16", 600011)])
def test_bonus_draw_over_many_row_tiles(dtype, V):
    """Target row gamma spans more than 64 of its 16 KiB tiles, so the draw
    locates its tile with the workgroup-wide scan; drafts equal to the
    target rows make every draft accepted."""
    x = W.small_case(3, 2, V, dtype, seed=93)
    x.draft[:] = x.target[:, :2]
    compare(x, run_gpu(x), run_oracle(x), label=f"many row tiles {dtype}")


@pytest.mark.parametrize("dtype,V", [("bf16", 131072), ("bf16", 131073), ("f16", 131071), ("f32", 65536),
                                     ("f32", 65537)])
def test_bonus_draw_at_the_one_wave_limit(dtype, V):
    """Target row gamma in 16 tiles of 16 KiB (64 quarter masses: one wave
    does the draw) or 17 (68: the workgroup does it), with and without a
    ragged last tile; every draft accepted, so every element draws from that
    row."""
    x = W.small_case(8, 2, V, dtype, seed=95)
    x.draft[:] = x.target[:, :2]
    g = run_gpu(x)
    assert np.all(g.accepted_len == 2), g.accepted_len
    compare(x, g, run_oracle(x), label=f"one-wave limit {dtype} V={V}")


@pytest.mark.parametrize("ab", [10.0, 1e3, 1e4, 1e5])
def test_sigmoid_scaling_constants(ab):
    x = W.small_case(16, 10, 50272, "f16", mode="sigmoid", seed=51, temperature=0.7, alpha=-ab, beta=ab)
    g = run_gpu(x)
    assert np.all(np.isfinite(g.tau))
    compare(x, g, run_oracle(x), label=f"sigmoid +-{ab:g}")


def test_sigmoid_zero_residual_fallback():
    # p_hat <= q_hat everywhere in row 0 and the draft rejected: draw from p_hat_0
    x = W.small_case(4, 2, 333, "f32", mode="sigmoid", seed=61, alpha=-10.0, beta=10.0)
    x.draft[:, 0, :] = x.target[:, 0, :] + 1.0
    x.uniforms[:, 0] = 0.999999
    g = run_gpu(x)
    o = run_oracle(x)
    assert np.all(o.fallback)
    compare(x, g, o, label="fallback")


@pytest.mark.parametrize("idx", range(9))
def test_golden_examples_on_gpu(golden_examples, idx):
    ex = golden_examples[idx]
    draft, target, tokens, uniforms = example_arrays(ex, dtype=np.float32)
    x = W.Inputs(draft, target, tokens, uniforms.astype(np.float32), "f32", ex["mode"], ex["temperature"],
                 ex["alpha"], ex["beta"])
    g = run_gpu(x)
    assert int(g.accepted_len[0]) == ex["expect"]["accepted_len"], ex["name"]
    assert int(g.next_token[0]) == ex["expect"]["next_token"], ex["name"]


def test_deterministic_and_workspace_reuse():
    big = W.small_case(16, 8, 40000, "bf16", seed=71)
    small = W.small_case(3, 2, 999, "bf16", seed=72)
    ws = binding.new_workspace(16, 8, 40000, torch.bfloat16, "cuda")
    first = run_gpu(big, workspace=ws)
    for _ in range(20):
        again = run_gpu(big, workspace=ws)
        assert np.array_equal(first.accepted_len, again.accepted_len)
        assert np.array_equal(first.next_token, again.next_token)
        assert np.array_equal(first.tau, again.tau) and np.array_equal(first.weights, again.weights)
    assert binding.workspace_bytes(3, 2, 999, torch.bfloat16) <= ws.numel()
    compare(small, run_gpu(small, workspace=ws), run_oracle(small), label="reuse smaller")
    compare(big, run_gpu(big, workspace=ws), run_oracle(big), label="reuse bigger again")
    # every call hands the workspace back zero-filled: ticket counter reset,
    # published words cleared, no timed-out wait
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(ws)) == 0


@pytest.mark.parametrize("mode", ["exact", "sigmoid"])
def test_workspace_returns_to_zero(mode):
    x = W.small_case(5, 4, 7001, "f16", mode=mode, seed=81, alpha=-1e3, beta=1e3)
    x.tokens[1, 0] = -1                        # a sentinel row must clean up too
    ws = binding.new_workspace(5, 4, 7001, torch.float16, "cuda")
    for _ in range(3):
        run_gpu(x, workspace=ws)
        torch.cuda.synchronize()
        assert int(torch.count_nonzero(ws)) == 0


def test_gpu_emits_target_distribution_tiny_vocab():
    """10^6 seeded steps through the GPU with fixed rows: the token emitted at
    each position is distributed as p (3-sigma per category)."""
    gamma, V, n = 3, 8, 1_000_000
    g = np.random.Generator(np.random.PCG64(808))
    z_p = g.normal(0, 1.5, size=(gamma + 1, V)).astype(np.float32)
    z_q = (z_p[:gamma] + g.normal(0, 1.0, size=(gamma, V))).astype(np.float32)
    tokens = np.stack([W.gumbel_max_tokens(g, np.broadcast_to(z_q[c].astype(np.float64), (n, V)), 1.0)
                       for c in range(gamma)], axis=1)
    u = np.minimum(g.random((n, gamma + 1)).astype(np.float32), W.UNIFORM_MAX)
    x = W.Inputs(np.ascontiguousarray(np.broadcast_to(z_q, (n, gamma, V))),
                 np.ascontiguousarray(np.broadcast_to(z_p, (n, gamma + 1, V))), tokens, u, "f32", "exact", 1.0,
                 -1e4, 1e4)
    acc, nxt = run_gpu(x, probe=False)
    assert np.all(acc >= 0)
    P = np.exp(z_p.astype(np.float64) - z_p.max(-1, keepdims=True))
    P /= P.sum(-1, keepdims=True)
    for c in range(gamma + 1):
        reached = acc >= c
        emitted = np.where(acc[reached] > c, tokens[reached, min(c, gamma - 1)] if c < gamma else -1,
                           nxt[reached])
        m = emitted.size
        counts = np.bincount(emitted, minlength=V)
        sigma = np.sqrt(m * P[c] * (1 - P[c]))
        assert np.all(np.abs(counts - m * P[c]) <= 3 * sigma), (c, counts, m * P[c], sigma)


@pytest.mark.parametrize("alpha,beta,seed", [(-10.0, 10.0, 31), (-3.0, 3.0, 32)])
def test_gpu_sigmoid_first_token_law_tiny_vocab(alpha, beta, seed):
    """10^6 seeded steps of the sigmoid mode through the GPU with fixed rows
    and drafts x ~ q (the draft's softmax): the first emitted token has the
    law q tau_hat + (1 - sum q tau_hat) a_hat / b_hat of the approximate test
    and residual of Sec. 3.2.2 (the same closed form as the oracle's CPU
    check), within a Bonferroni bar of 1e-4 family-wise.  Seeds fixed in
    advance."""
    gamma, V, n, T = 2, 6, 1_000_000, 1.0
    g = np.random.Generator(np.random.PCG64(seed))
    z_p = g.normal(0, 8, size=(gamma + 1, V)).astype(np.float32)
    z_q = (z_p[:gamma] + g.normal(0, 8, size=(gamma, V))).astype(np.float32)
    tokens = np.stack([W.gumbel_max_tokens(g, np.broadcast_to(z_q[c].astype(np.float64), (n, V)), T)
                       for c in range(gamma)], axis=1)
    u = np.minimum(g.random((n, gamma + 1)).astype(np.float32), W.UNIFORM_MAX)
    x = W.Inputs(np.ascontiguousarray(np.broadcast_to(z_q, (n, gamma, V))),
                 np.ascontiguousarray(np.broadcast_to(z_p, (n, gamma + 1, V))), tokens, u, "f32", "sigmoid", T,
                 alpha, beta)
    acc, nxt = run_gpu(x, probe=False)
    assert np.all(acc >= 0)
    first = np.where(acc >= 1, tokens[:, 0], nxt)
    zp0, zq0 = z_p[0].astype(np.float64), z_q[0].astype(np.float64)
    ph = scipy.special.expit((zp0 / T - alpha) / (beta - alpha))
    qh = scipy.special.expit((zq0 / T - alpha) / (beta - alpha))
    q = scipy.special.softmax(zq0 / T)
    tau = np.minimum(1.0, ph / qh)
    resid = np.maximum(0.0, ph - qh)
    law = q * tau + (1.0 - np.sum(q * tau)) * resid / resid.sum()
    assert abs(law.sum() - 1.0) < 1e-12
    k = int(np.sum(law > 0))
    nsigma = float(scipy.stats.norm.isf(1e-4 / (2 * k)))
    counts = np.bincount(first, minlength=V)
    sigma = np.sqrt(n * law * (1 - law))
    dev = np.abs(counts - n * law)
    print(f"[sigmoid law] alpha={alpha}: max deviation {np.max(dev / np.maximum(sigma, 1e-12)):.2f} sigma "
          f"(bar {nsigma:.2f})", flush=True)
    assert np.all(dev <= nsigma * sigma + 1e-9), (counts, n * law, sigma)
    assert np.all(counts[law == 0] == 0)


# --- seeded random shapes ------------------------------------------------------

def test_randomized_shapes():
    """60 seeded random cases: batch 1-9, gamma 1-24, V 1-6000, every dtype and
    mode, temperature 0.3-2, noise from near-identical to unrelated rows, some
    with top-k masks, some ragged."""
    rng = np.random.default_rng(20261202)
    for case in range(60):
        B = int(rng.integers(1, 10))
        g = int(rng.integers(1, 25))
        V = int(rng.choice([1, 2, 3, 17, 64, 255, 1000, 2049, 4096, 5999]))
        dtype = str(rng.choice(["f32", "f16", "bf16"]))
        mode = str(rng.choice(["exact", "sigmoid"]))
        T = float(rng.choice([0.3, 0.7, 1.0, 2.0]))
        noise = float(rng.choice([0.01, 0.2, 1.0, 4.0]))
        top_k = int(rng.choice([0, 0, 0, 1, 5, 50]))
        ab = float(rng.choice([10.0, 1e3, 1e4]))
        x = W.small_case(B, g, V, dtype, mode=mode, seed=5000 + case, temperature=T, noise_scale=noise,
                         top_k=top_k, alpha=-ab, beta=ab)
        label = f"case {case}: B={B} g={g} V={V} {dtype} {mode} T={T} noise={noise} k={top_k}"
        if case % 4 == 3:
            gam = rng.integers(1, g + 1, size=B).astype(np.int32)
            d, t, tok, u = binding.to_device(x, "cuda")
            acc, nxt = binding.verify(d, t, tok, u, mode=mode, temperature=T, alpha=-ab, beta=ab,
                                      gammas=torch.from_numpy(gam).to("cuda"))
            torch.cuda.synchronize()
            with np.errstate(all="ignore"):
                o = oracle.verify_ragged(x.draft, x.target, x.tokens, x.uniforms, gam, dtype=dtype, mode=mode,
                                         temperature=T, alpha=-ab, beta=ab)
            ok = ~o.flagged(1e-6)
            assert np.array_equal(acc.cpu().numpy()[ok], o.accepted_len[ok]), label
            assert np.array_equal(nxt.cpu().numpy()[ok], o.next_token[ok]), label
        else:
            compare(x, run_gpu(x), run_oracle(x), label=label)


def test_determinism_at_the_headline_shape():
    """1000 back-to-back calls on the headline workload give bit-identical
    outputs (every reduction has a fixed order; no float atomics)."""
    x = W.generate(W.WORKLOADS["exact_b64_g8_v128256_bf16"])
    d, t, tok, u = binding.to_device(x, "cuda")
    ws = binding.new_workspace(x.batch, x.gamma, x.vocab, d.dtype, "cuda")
    a0, n0 = binding.verify(d, t, tok, u, workspace=ws)
    a0, n0 = a0.clone(), n0.clone()
    acc = torch.empty_like(a0)
    nxt = torch.empty_like(n0)
    same = torch.ones((), dtype=torch.bool, device="cuda")
    for _ in range(1000):
        binding.verify(d, t, tok, u, accepted_len=acc, next_token=nxt, workspace=ws)
        same &= (acc == a0).all() & (nxt == n0).all()
    torch.cuda.synchronize()
    assert bool(same)
    assert int(torch.count_nonzero(ws)) == 0


def test_decisions_do_not_depend_on_the_batch_tiling():
    """The same batch elements verified inside the full batch (B = 64: 32 KiB
    chunks, bonus tiles), as a batch of 8 and one by one (B = 1: one vector
    per thread) take different chunkings and layouts; the decisions agree
    everywhere the oracle does not flag a threshold."""
    w = W.WORKLOADS["exact_b64_g8_v128256_bf16"]
    x = W.generate(w)
    sub = W.generate(w, batch_indices=range(8))
    o = run_oracle(sub)
    ok = ~o.flagged(1e-6)
    full = run_gpu(x, probe=False)
    eight = run_gpu(sub, probe=False)
    singles = [run_gpu(W.generate(w, batch_indices=range(b, b + 1)), probe=False) for b in range(8)]
    one_acc = np.array([s[0][0] for s in singles])
    one_nxt = np.array([s[1][0] for s in singles])
    for acc, nxt in ((full[0][:8], full[1][:8]), eight, (one_acc, one_nxt)):
        assert np.array_equal(acc[ok], o.accepted_len[ok])
        assert np.array_equal(nxt[ok], o.next_token[ok])
