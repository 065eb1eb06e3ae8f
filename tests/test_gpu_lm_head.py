"""Embedding and output head + cross-entropy kernels against the oracle,
through the C ABI, at small shapes and at the LM workload's full shape
(64 windows x 256 positions, width 512, 256 byte values, Zipf tokens)."""
import numpy as np
import pytest
import torch

from oracle import lm_head
from paper_2609_18145_amd import hcmix, inputs
from tests.util import to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


@pytest.mark.parametrize("rows,width,vocab", [(100, 64, 256), (16384, 512, 256), (40000, 128, 37)])
def test_embedding_forward_is_an_exact_gather(rows, width, vocab):
    print(f"case: embedding forward rows={rows} width={width} vocab={vocab}", flush=True)
    rng = np.random.default_rng(rows)
    table = inputs.round_bf16(rng.standard_normal((vocab, width)).astype(np.float32))
    tokens = rng.integers(0, vocab, rows)
    tokens[::97] = vocab          # out of range: zero rows
    tokens[5::101] = -3
    x = hcmix.embedding_forward(to_dev(table, "bf16"), i32(tokens))
    torch.cuda.synchronize()
    want = np.zeros((rows, width), dtype=np.float32)
    ok = (tokens >= 0) & (tokens < vocab)
    want[ok] = table[tokens[ok]]
    assert np.array_equal(to_host(x), want)


@pytest.mark.parametrize("rows,width,vocab,zipf", [(300, 64, 16, False), (16384, 512, 256, True),
                                                    (40000, 128, 37, False)])
def test_embedding_backward_matches_oracle_and_repeats(rows, width, vocab, zipf):
    print(f"case: embedding backward rows={rows} width={width} vocab={vocab}", flush=True)
    rng = np.random.default_rng(rows + 1)
    if zipf:
        tokens = inputs.zipf_byte_tokens(rng, (rows,))
    else:
        tokens = rng.integers(0, vocab, rows)
    tokens[7::131] = vocab + 5    # skipped
    dx = inputs.round_bf16(rng.standard_normal((rows, width)).astype(np.float32))
    t, g = i32(tokens), to_dev(dx, "bf16")
    a = hcmix.embedding_backward(t, g, vocab)
    b = hcmix.embedding_backward(t, g, vocab)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    ok = tokens < vocab
    ref = lm_head.embedding_backward(tokens[ok], dx[ok], vocab)
    err = np.abs(to_host(a) - ref).max() / max(np.abs(ref).max(), 1e-30)
    print(f"  max err / max |ref| {err:.2e}", flush=True)
    assert err <= 1e-5
    base = a.clone()
    hcmix.embedding_backward(t, g, vocab, dtable=a, accumulate=True)
    torch.cuda.synchronize()
    assert torch.equal(a, 2 * base)


@pytest.mark.parametrize("rows,width,vocab", [(200, 64, 256), (1000, 512, 256), (130, 128, 96),
                                              (64, 192, 32)])
def test_head_cross_entropy_matches_oracle(rows, width, vocab):
    print(f"case: head + CE rows={rows} width={width} vocab={vocab}", flush=True)
    rng = np.random.default_rng(rows + vocab)
    x = inputs.round_bf16(rng.standard_normal((rows, width)).astype(np.float32))
    w = inputs.round_bf16((rng.standard_normal((vocab, width)) / np.sqrt(width)).astype(np.float32))
    bias = (rng.standard_normal(vocab) * 0.3).astype(np.float32)
    targets = rng.integers(0, vocab, rows)
    args = (to_dev(x, "bf16"), to_dev(w, "bf16"), torch.from_numpy(bias).cuda(), i32(targets),
            1.0 / rows)
    loss, d, db = hcmix.head_cross_entropy(*args, with_dbias=True)
    loss2, d2 = hcmix.head_cross_entropy(*args)             # without the bias gradient
    _, _, db2 = hcmix.head_cross_entropy(*args, with_dbias=True)
    torch.cuda.synchronize()
    r_loss, r_d = lm_head.head_cross_entropy(x, w, bias, targets, 1.0 / rows)
    e_loss = np.abs(to_host(loss) - r_loss).max()
    g, r = to_host(d), r_d
    e_d = (np.linalg.norm(g - r, axis=1) / np.linalg.norm(r, axis=1)).max()
    r_db = r_d.sum(axis=0)
    e_db = np.linalg.norm(to_host(db) - r_db) / np.linalg.norm(r_db)
    print(f"  loss abs err {e_loss:.2e}  dlogits row err {e_d:.2e}  dbias err {e_db:.2e}",
          flush=True)
    assert e_loss <= 1e-4
    assert e_d <= 2e-2
    assert e_db <= 1e-3
    assert torch.equal(loss, loss2) and torch.equal(d, d2) and torch.equal(db, db2)


def test_head_cross_entropy_full_lm_shape_sampled():
    """16384 rows (64 windows of 256), width 512, 256-way head: every loss, the
    bias gradient, and the gradient rows of windows 0 and 63, against the
    oracle."""
    rows, width, vocab = 16384, 512, 256
    rng = np.random.default_rng(9)
    x = inputs.round_bf16(rng.standard_normal((rows, width)).astype(np.float32))
    w = inputs.round_bf16((rng.standard_normal((vocab, width)) / np.sqrt(width)).astype(np.float32))
    bias = np.zeros(vocab, dtype=np.float32)
    targets = inputs.zipf_byte_tokens(rng, (rows,))
    loss, d, db = hcmix.head_cross_entropy(to_dev(x, "bf16"), to_dev(w, "bf16"),
                                           torch.from_numpy(bias).cuda(), i32(targets),
                                           1.0 / rows, with_dbias=True)
    torch.cuda.synchronize()
    r_loss, r_all = lm_head.head_cross_entropy(x, w, bias, targets, 1.0 / rows)
    assert np.abs(to_host(loss) - r_loss).max() <= 1e-4
    r_db = r_all.sum(axis=0)
    assert np.linalg.norm(to_host(db) - r_db) / np.linalg.norm(r_db) <= 1e-3
    for sl in (slice(0, 256), slice(rows - 256, rows)):
        _, r_d = lm_head.head_cross_entropy(x[sl], w, bias, targets[sl], 1.0 / rows)
        g = to_host(d)[sl]
        assert (np.linalg.norm(g - r_d, axis=1) / np.linalg.norm(r_d, axis=1)).max() <= 2e-2
