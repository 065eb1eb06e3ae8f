"""Embedding and output head + cross-entropy kernels against the oracle,
through the C ABI, at small shapes and at the LM workload's full shape
(64 windows x 256 positions, width 512, 256 byte values, Zipf tokens)."""
import numpy as np
import pytest
import torch

from oracle import lm_head
from paper_2609_18145_amd import hcmix, inputs
from tests.util import TOL, fro_rel_err, row_rel_err, to_dev, to_host

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
                                                    (40000, 128, 37, False), (3000, 1024, 6, False),
                                                    (70000, 64, 256, True)])
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


def test_whole_lm_step_replays_in_a_graph():
    """The LM step the default benchmark replays (embedding gather, the stack
    forward on the deferred path, head + cross-entropy with the bias gradient,
    the input gradient as a plain product, the stack backward, the embedding's
    scatter sum), captured from a side stream and replayed three times with
    eager work and synchronisation in between: every output of every replay
    bitwise equal to the eager step, and the loss against the oracle."""
    import oracle
    B, n, w, L, V = 4, 256, 256, 4, 256
    rows = B * n
    s = inputs.make_stack(batch=B, n=n, width=w, num_layers=L, causal=True, dtype="bf16", seed=71)
    rng = np.random.default_rng(72)
    table_np = inputs.round_bf16(rng.standard_normal((V, w)).astype(np.float32))
    head_np = inputs.round_bf16((rng.standard_normal((V, w)) / np.sqrt(w)).astype(np.float32))
    tokens_np = inputs.zipf_byte_tokens(rng, (rows,))
    targets_np = inputs.zipf_byte_tokens(rng, (rows,))
    print(f"case: LM step graph replay B={B} n={n} w={w} L={L} V={V}", flush=True)
    table, head_w = to_dev(table_np, "bf16"), to_dev(head_np, "bf16")
    head_b = torch.zeros(V, dtype=torch.float32, device="cuda")
    tokens, targets = i32(tokens_np), i32(targets_np)
    ws = [to_dev(a, "bf16") for a in s.w_self]
    wo = [to_dev(a, "bf16") for a in s.w_off]
    x0 = torch.empty(B, n, w, dtype=torch.bfloat16, device="cuda")
    outs = [torch.empty_like(x0) for _ in range(L)]
    dx0 = torch.empty_like(x0)
    gx = torch.empty(rows, w, dtype=torch.bfloat16, device="cuda")
    dws = [torch.empty((w, w), dtype=torch.float32, device="cuda") for _ in range(L)]
    dwo = [torch.empty((w, w), dtype=torch.float32, device="cuda") for _ in range(L)]
    loss = torch.empty(rows, dtype=torch.float32, device="cuda")
    dlog = torch.empty(rows, V, dtype=torch.bfloat16, device="cuda")
    dbias = torch.empty(V, dtype=torch.float32, device="cuda")
    dtable = torch.empty(V, w, dtype=torch.float32, device="cuda")
    stack_ws = hcmix.alloc_stack_workspace(B, n, w, L, torch.bfloat16, "cuda")
    head_ws = torch.empty(hcmix.load().hcmix_head_cross_entropy_workspace_bytes(rows, V),
                          dtype=torch.uint8, device="cuda")
    emb_ws = torch.empty(hcmix.load().hcmix_embedding_backward_workspace_bytes(rows, w, V),
                         dtype=torch.uint8, device="cuda")
    results = [x0, *outs, loss, dlog, dbias, gx, dx0, *dws, *dwo, dtable]

    def step():
        hcmix.embedding_forward(table, tokens, out=x0)
        xs = hcmix.stack_forward(x0, ws, wo, s.layers, True, outs=outs)
        hcmix.head_cross_entropy(xs[-1].view(rows, w), head_w, head_b, targets, 1.0 / rows,
                                 loss=loss, dlogits=dlog, dbias=dbias, workspace=head_ws)
        torch.matmul(dlog, head_w, out=gx)
        hcmix.stack_backward(xs, ws, wo, s.layers, gx.view(B, n, w), True, dx=dx0, dws=dws,
                             dwo=dwo, workspace=stack_ws)
        hcmix.embedding_backward(tokens, dx0, V, dtable=dtable, workspace=emb_ws)

    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        step()
        torch.cuda.synchronize()
        ref = [t.clone() for t in results]
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            step()
    # the eager step against the oracle's forward: the loss of every row
    xs_ref = oracle.stack_forward(table_np[tokens_np].reshape(B, n, w), s.w_self, s.w_off,
                                  s.layers, True)
    r_loss, _ = lm_head.head_cross_entropy(to_host(ref[L]).reshape(rows, w), head_np,
                                           np.zeros(V), targets_np, 1.0 / rows)
    assert np.abs(to_host(ref[L + 1]) - r_loss).max() <= 1e-3
    rel = (np.linalg.norm(to_host(ref[L]) - xs_ref[-1]) / np.linalg.norm(xs_ref[-1]))
    assert rel <= 2e-2
    for rep in range(3):
        for t in results:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(results, ref)):
            assert torch.equal(a, b), f"replay {rep}: output {k} differs from the eager step"
        print(f"  replay {rep} bitwise equal", flush=True)


@pytest.mark.parametrize("rows,width,vocab", [(16384, 512, 256), (1000, 192, 96), (200, 64, 32),
                                              (130, 1024, 288), (77, 128, 64)])
def test_head_backward_matches_oracle_and_repeats(rows, width, vocab):
    """gx = dlogits W and dW = dlogits^T x against the oracle on the same bf16
    operands (one full LM shape, ragged rows, vocabulary and width tiles that
    do not fill 128); dW bitwise-repeatable and accumulating; each output alone
    equals the pair's."""
    print(f"case: head backward rows={rows} width={width} vocab={vocab}", flush=True)
    rng = np.random.default_rng(rows + vocab)
    x = inputs.round_bf16(rng.standard_normal((rows, width)).astype(np.float32))
    w = inputs.round_bf16((rng.standard_normal((vocab, width)) / np.sqrt(width)).astype(np.float32))
    d = inputs.round_bf16((rng.standard_normal((rows, vocab)) / rows).astype(np.float32))
    xg, wg, dg = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(d, "bf16")
    gx, dw = hcmix.head_backward(xg, wg, dg)
    gx2, dw2 = hcmix.head_backward(xg, wg, dg)
    torch.cuda.synchronize()
    want_gx, want_dw = lm_head.head_backward(x, w, d)
    e_gx = row_rel_err(to_host(gx), want_gx)
    e_dw = fro_rel_err(to_host(dw), want_dw)
    print(f"  gx row err {e_gx:.2e}, dW err {e_dw:.2e}", flush=True)
    assert e_gx <= TOL["bf16"]
    assert e_dw <= 1e-4
    assert torch.equal(gx, gx2) and torch.equal(dw, dw2)
    only_gx, none_dw = hcmix.head_backward(None, wg, dg, with_dw=False)   # x unused
    none_gx, only_dw = hcmix.head_backward(xg, wg, dg, with_gx=False)
    base = dw.clone()
    hcmix.head_backward(xg, wg, dg, dw=dw, with_gx=False, accumulate=True)
    torch.cuda.synchronize()
    assert none_dw is None and none_gx is None
    assert torch.equal(only_gx, gx) and torch.equal(only_dw, base)
    assert torch.equal(dw, base + base)
