"""The whole step captured into a HIP graph: every replay reproduces the eager
result bit for bit, with eager work and synchronisations between replays (the
library enqueues no memset, so nothing in the graph depends on one)."""

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _cuda(a):
    import torch

    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("fused", [False, True])  # selection and loss in one call
@pytest.mark.parametrize("T", [700, 6000])  # one-workgroup and many-workgroup loss
def test_graph_replays_match_eager(T, fused):
    import torch

    import paper_2509_23866_amd as dart

    V, S = 2048, 30
    rng = np.random.default_rng(T)
    logits = torch.from_numpy(rng.normal(0, 3, (T, V)).astype(np.float32)).cuda().to(torch.bfloat16)
    target = _cuda(rng.integers(0, V, T).astype(np.int32))
    off = _cuda(np.r_[0, np.sort(rng.choice(np.arange(1, T), S - 1, replace=False)), T].astype(np.int32))
    logp0, _, _ = dart.dart_tok_stats(logits, target)
    lp_old = logp0 + _cuda(rng.normal(0, 0.05, T).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, T).astype(np.float32))
    adv = _cuda(rng.normal(0, 1, T).astype(np.float32))

    def buffers():
        f = lambda n: torch.empty(n, dtype=torch.float32, device="cuda")  # noqa: E731
        return dict(logp=f(T), ent=f(T), lse=f(T), sh=f(S),
                    mask=torch.empty(S, dtype=torch.uint8, device="cuda"),
                    nk=torch.empty(1, dtype=torch.int32, device="cuda"),
                    loss=torch.empty(1, dtype=torch.float64, device="cuda"), coef=f(T), st=f(4),
                    ws=torch.empty(dart.dart_tis_loss_workspace_bytes(T), dtype=torch.uint8,
                                   device="cuda"),
                    dz=torch.empty_like(logits))

    def step(b, s=None):
        dart.dart_tok_stats(logits, target, b["logp"], b["ent"], b["lse"], stream=s)
        if fused:
            dart.dart_select_tis_loss_fwd(b["ent"], b["logp"], lp_old, lp_roll, adv, off, 0.8,
                                          0.2, 0.28, 2.0, b["sh"], b["mask"], b["nk"], b["loss"],
                                          b["coef"], b["st"], stream=s, workspace=b["ws"])
        else:
            dart.dart_step_select(b["ent"], off, 0.8, b["sh"], b["mask"], b["nk"], stream=s)
            dart.dart_tis_loss_fwd(b["logp"], lp_old, lp_roll, adv, off, b["mask"], 0.2, 0.28,
                                   2.0, b["loss"], b["coef"], b["st"], stream=s, workspace=b["ws"])
        dart.dart_tis_grad(logits, target, b["logp"], b["lse"], b["coef"], b["dz"], stream=s)

    eager = buffers()
    step(eager)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items() if k != "ws"}

    gb = buffers()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(gb, side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        step(gb, side)
    for rep in range(4):
        for v in gb.values():
            v.fill_(0)  # stale results must not survive into the check
        g.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(gb[k].view(torch.uint8), v.view(torch.uint8)), (rep, k)
        step(eager)  # eager work between replays
        torch.cuda.synchronize()


def test_synchronising_mode_refused_under_capture(monkeypatch):
    """DART_CHECK=1 waits for the host: on a stream that is being captured a
    call returns DART_ERR_UNSUPPORTED with nothing enqueued, and the capture
    goes on (a statistics call captured after it replays to the eager bits)."""
    import torch

    import paper_2509_23866_amd as dart

    T, V = 64, 300
    rng = np.random.default_rng(5)
    y = _cuda(rng.integers(0, V, T).astype(np.int32))
    logits = torch.from_numpy(rng.normal(0, 3, (T, V)).astype(np.float32)).cuda()
    out = [torch.empty(T, dtype=torch.float32, device="cuda") for _ in range(3)]
    ref = dart.dart_tok_stats(logits, y)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    codes = []
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        monkeypatch.setenv("DART_CHECK", "1")
        try:
            dart.dart_tok_stats(logits, y, *out, stream=side)
        except dart.DartError as e:
            codes.append(e.code)
        monkeypatch.setenv("DART_CHECK", "0")
        dart.dart_tok_stats(logits, y, *out, stream=side)
    assert codes == [dart.DART_ERR_UNSUPPORTED]
    for _ in range(2):
        for o in out:
            o.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, r in zip(out, ref):
            assert torch.equal(o, r)


@pytest.mark.parametrize("rows,cols,bf16", [(64, 300, False), (32, 128, True)])
def test_lmhead_skip_rows_graph_follows_the_device_count(rows, cols, bf16):
    """The row-skipping LM-head backward reads the kept-row count on the
    device, so it captures into a graph; replays after the coefficients change
    in place (more, fewer, all and no rows kept) give the bits of an eager call
    on the new coefficients, in row blocks of 64 or 32 and vocabulary blocks."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V = 150, 64, 300
    rng = np.random.default_rng(21)
    h = torch.from_numpy(rng.normal(0, 1, (T, d)).astype(np.float32)).cuda().to(torch.bfloat16)
    w = torch.from_numpy(rng.normal(0, 0.3, (V, d)).astype(np.float32)).cuda().to(torch.bfloat16)
    y = _cuda(rng.integers(0, V, T).astype(np.int32))
    logp, _, lse = dart.dart_lmhead_tok_stats(h, w, y)
    flags = dart.DART_LMHEAD_SKIP_ZERO_ROWS | (dart.DART_LMHEAD_BF16_GRADS if bf16 else 0)
    gdt = torch.bfloat16 if bf16 else torch.float32
    coef = torch.empty(T, dtype=torch.float32, device="cuda")
    dh = torch.empty((T, d), dtype=gdt, device="cuda")
    dw = torch.empty((V, d), dtype=gdt, device="cuda")
    ws = torch.empty(dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, flags),
                     dtype=torch.uint8, device="cuda")
    patterns = [np.where(rng.random(T) < p, 0.0, rng.uniform(-1e-2, 1e-2, T)) for p in (0.3, 0.8)]
    patterns += [np.full(T, 3e-3), np.zeros(T)]

    def call(s):
        dart.dart_lmhead_backward_ex(h, w, y, lse, logp, coef, chunk_rows=rows, chunk_cols=cols,
                                     flags=flags, dhidden=dh, dweight=dw, workspace=ws, stream=s)

    coef.copy_(torch.from_numpy(patterns[0].astype(np.float32)))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        call(side)
    torch.cuda.synchronize()
    for pat in patterns + patterns[:1]:
        coef.copy_(torch.from_numpy(pat.astype(np.float32)))
        torch.cuda.synchronize()
        call(torch.cuda.current_stream())
        torch.cuda.synchronize()
        eager = (dh.clone(), dw.clone())
        dh.view(torch.uint8).fill_(0x7F)
        dw.view(torch.uint8).fill_(0x7F)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(dh.view(torch.uint8), eager[0].view(torch.uint8))
        assert torch.equal(dw.view(torch.uint8), eager[1].view(torch.uint8))
        zero = torch.from_numpy(pat == 0.0).cuda()
        assert torch.all(dh[zero] == 0)
        if not pat.any():  # no row kept: dweight is exactly zero
            assert torch.all(dw == 0)


@pytest.mark.parametrize("rows,cols,bf16", [(256, 300, False), (100, 128, True)])
def test_lmhead_step_graph_replays_match_eager(rows, cols, bf16):
    """The fused LM-head step (statistics, selection, loss, blocked backward
    with its GEMMs) captured once: every replay gives the eager bits,
    with eager work and synchronisations between replays."""
    import torch

    import paper_2509_23866_amd as dart

    T, d, V, S = 256, 64, 300, 8
    rng = np.random.default_rng(11)
    h = torch.from_numpy(rng.normal(0, 1, (T, d)).astype(np.float32)).cuda().to(torch.bfloat16)
    w = torch.from_numpy(rng.normal(0, 0.3, (V, d)).astype(np.float32)).cuda().to(torch.bfloat16)
    y = _cuda(rng.integers(0, V, T).astype(np.int32))
    off = _cuda(np.r_[0, np.sort(rng.choice(np.arange(1, T), S - 1, replace=False)), T].astype(np.int32))
    lp_old = _cuda(rng.normal(-5, 1, T).astype(np.float32))
    lp_roll = lp_old + _cuda(rng.normal(0, 0.1, T).astype(np.float32))
    adv = _cuda(rng.normal(0, 1, T).astype(np.float32))
    flags = dart.DART_LMHEAD_BF16_GRADS if bf16 else 0
    gdt = torch.bfloat16 if bf16 else torch.float32
    f = lambda n: torch.empty(n, dtype=torch.float32, device="cuda")  # noqa: E731
    b = dict(logp=f(T), ent=f(T), lse=f(T), sh=f(S),
             mask=torch.empty(S, dtype=torch.uint8, device="cuda"),
             nk=torch.empty(1, dtype=torch.int32, device="cuda"),
             loss=torch.empty(1, dtype=torch.float64, device="cuda"), coef=f(T), st=f(4),
             sws=torch.empty(dart.dart_lmhead_stats_workspace_bytes(T, V), dtype=torch.uint8,
                             device="cuda"),
             lws=torch.empty(dart.dart_tis_loss_workspace_bytes(T), dtype=torch.uint8, device="cuda"),
             bws=torch.empty(dart.dart_lmhead_backward_ex_workspace_bytes(T, d, V, rows, cols, flags),
                             dtype=torch.uint8, device="cuda"),
             dh=torch.empty((T, d), dtype=gdt, device="cuda"),
             dw=torch.empty((V, d), dtype=gdt, device="cuda"))

    def step(s):
        dart.dart_lmhead_tok_stats(h, w, y, b["logp"], b["ent"], b["lse"], workspace=b["sws"],
                                   stream=s)
        dart.dart_step_select(b["ent"], off, 0.6, b["sh"], b["mask"], b["nk"], stream=s)
        dart.dart_tis_loss_fwd(b["logp"], lp_old, lp_roll, adv, off, b["mask"], 0.2, 0.28, 2.0,
                               loss=b["loss"], tok_coef=b["coef"], stats=b["st"],
                               workspace=b["lws"], stream=s)
        dart.dart_lmhead_backward_ex(h, w, y, b["lse"], b["logp"], b["coef"], chunk_rows=rows,
                                     chunk_cols=cols, flags=flags, dhidden=b["dh"],
                                     dweight=b["dw"], workspace=b["bws"], stream=s)

    keys = ("logp", "ent", "lse", "mask", "loss", "coef", "dh", "dw")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(side)
    torch.cuda.synchronize()
    eager = {k: b[k].clone() for k in keys}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        step(side)
    for _ in range(3):
        for k in keys:
            b[k].view(torch.uint8).fill_(0x7F)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in keys:
            assert torch.equal(b[k].view(torch.uint8), eager[k].view(torch.uint8)), k
