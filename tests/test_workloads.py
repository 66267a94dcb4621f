"""The seeded input generator: shapes, determinism, storage rounding, draft law."""
import numpy as np
import pytest
import scipy.special
import torch

from paper_2406_11016_amd import workloads as W


def test_named_workloads_shapes():
    expect = {
        "exact_b1_g5_v51865_f32": (1, 5, 51865, "f32", "exact"),
        "exact_b1_g10_v32000_f16": (1, 10, 32000, "f16", "exact"),
        "exact_b16_g5_v51865_f32": (16, 5, 51865, "f32", "exact"),
        "exact_b64_g8_v128256_bf16": (64, 8, 128256, "bf16", "exact"),
        "sigmoid_b32_g10_v50272_f16_t0.7": (32, 10, 50272, "f16", "sigmoid"),
    }
    for name, (B, g, V, dt, mode) in expect.items():
        w = W.WORKLOADS[name]
        assert (w.batch, w.gamma, w.vocab, w.dtype, w.mode) == (B, g, V, dt, mode)
    assert W.WORKLOADS[W.HEADLINE].logit_bytes == 279_085_056


def test_generate_small_and_subset_determinism():
    w = W.WORKLOADS["exact_b16_g5_v51865_f32"].with_(vocab=1000)
    a = W.generate(w)
    assert a.draft.shape == (16, 5, 1000) and a.target.shape == (16, 6, 1000)
    assert a.draft.dtype == np.float32 and a.tokens.dtype == np.int32
    assert a.uniforms.shape == (16, 6) and a.uniforms.dtype == np.float32
    assert np.all((a.tokens >= 0) & (a.tokens < 1000))
    assert np.all((a.uniforms >= 0) & (a.uniforms <= W.UNIFORM_MAX))
    b = W.generate(w, batch_indices=range(5, 9))
    assert np.array_equal(a.draft[5:9], b.draft) and np.array_equal(a.target[5:9], b.target)
    assert np.array_equal(a.tokens[5:9], b.tokens) and np.array_equal(a.uniforms[5:9], b.uniforms)
    c = W.generate(w)
    assert np.array_equal(a.target, c.target)


def test_target_is_draft_plus_noise():
    w = W.WORKLOADS["exact_b1_g10_v32000_f16"].with_(vocab=4096)
    x = W.generate(w)
    d = x.target[:, :10].astype(np.float64) - x.draft.astype(np.float64)
    assert abs(d.std() - 1.0) < 0.05 and abs(x.draft.astype(np.float64).std() - 3.0) < 0.1


def test_bf16_rounding_matches_torch():
    v = np.random.default_rng(3).standard_t(3, size=100_000) * 2.0
    v = np.concatenate([v, [0.0, -0.0, 1e-40, 3.0e38, 1.00390625, 1.01171875]])
    ours = W.encode_bf16(v)
    ref = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(W.decode_bf16(ours), torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_gumbel_max_draws_from_softmax():
    g = np.random.Generator(np.random.PCG64(5))
    z = np.array([1.0, -0.5, 2.0, 0.0, -3.0])
    n = 400_000
    x = W.gumbel_max_tokens(g, np.broadcast_to(z, (n, 5)), 0.7)
    p = scipy.special.softmax(z / 0.7)
    counts = np.bincount(x, minlength=5)
    assert np.all(np.abs(counts - n * p) < 4 * np.sqrt(n * p * (1 - p)))


@pytest.mark.slow
def test_headline_workload_generates():
    w = W.WORKLOADS[W.HEADLINE]
    x = W.generate(w, batch_indices=range(2))
    assert x.draft.dtype == np.uint16 and x.draft.shape == (2, 8, 128256)
    vals = W.decode_bf16(x.target).astype(np.float64)
    assert np.isfinite(vals).all() and vals.max() > 20   # heavy tails


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_top_k_mask_keeps_the_k_largest(dtype):
    x = W.small_case(3, 4, 500, dtype, seed=5, top_k=7)
    full = W.small_case(3, 4, 500, dtype, seed=5)
    for masked, raw in ((x.draft, full.draft), (x.target, full.target)):
        m = W.stored_as_float64(masked, dtype)
        r = W.stored_as_float64(raw, dtype)
        keep = np.isfinite(m)
        assert np.all(keep.sum(axis=-1) == 7)
        assert np.all(m[keep] == r[keep])                              # kept values unchanged
        assert np.all(np.isneginf(m[~keep]))
        kth = np.sort(r, axis=-1)[..., -7]
        assert np.all(np.where(keep, r, np.inf).min(axis=-1) >= kth)   # the kept ones are the largest
    # drafted tokens are drawn from the masked draft rows
    d = W.stored_as_float64(x.draft, dtype)
    assert np.all(np.isfinite(np.take_along_axis(d, x.tokens[..., None].astype(np.int64), axis=-1)))
