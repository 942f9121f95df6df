"""The traffic-shape kernel (synth/synth.hip) that bench.py uses for the
bandwidth ceiling of a row set: it must touch exactly the coordinates it is
given, write back in-place rows unchanged, and fill write-only rows with the
XOR of what it read."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _words_f32(x):
    """(n,) fp32 tensor -> (n/4, 4) uint32 words per 4-coordinate group."""
    return x.cpu().numpy().view(np.uint32).reshape(-1, 4)


def _words_bf16(x):
    """(n,) bf16 tensor -> (n/4, 2) uint32 words (two bf16 per word, low first)."""
    h = x.view(torch.int16).cpu().numpy().view(np.uint16).astype(np.uint32).reshape(-1, 2)
    return (h[:, 0] | (h[:, 1] << 16)).reshape(-1, 2)


def test_shape_rows_in_place_keep_bits_and_pads():
    from synth.device import ShapePass, ShapeRow
    dev = torch.device("cuda:0")
    P, ld = 4 * 1024 * 3 + 8, 16384  # several blocks and a partly used last block
    g = torch.randn((3, ld), device=dev)
    b = torch.randn((2, ld), device=dev).to(torch.bfloat16)
    wo = torch.full((2, ld), 7.0, device=dev)
    g0, b0 = g.clone(), b.clone()
    rows = [ShapeRow(g, 0), ShapeRow(g, ld, write=True), ShapeRow(b, 0, write=True),
            ShapeRow(g, 2 * ld, write=True), ShapeRow(b, ld),
            ShapeRow(wo, 0, read=False), ShapeRow(wo, ld, read=False)]
    assert ShapePass(rows, P).bytes == P * (4 * 3 + 2 * 2 + 4 * 2 + 2 * 1 + 4 * 2)
    acc = np.zeros(P // 4, dtype=np.uint32)
    for r in range(3):
        acc ^= np.bitwise_xor.reduce(_words_f32(g[r, :P]), axis=1)
    for r in range(2):
        acc ^= np.bitwise_xor.reduce(_words_bf16(b[r, :P]), axis=1)
    for batch, xcd, threads in ((8, False, 256), (16, False, 256), (8, True, 256),
                                (16, True, 64), (8, False, 1024), (8, True, 128)):
        wo.fill_(7.0)
        ShapePass(rows, P, xcd=xcd, batch=batch, threads=threads).launch()
        torch.cuda.synchronize()
        assert torch.equal(g.view(torch.int32), g0.view(torch.int32))
        assert torch.equal(b.view(torch.int16), b0.view(torch.int16))
        for j in range(2):
            got = _words_f32(wo[j, :P])
            assert np.array_equal(got, np.repeat(acc[:, None], 4, axis=1)), \
                (batch, xcd, threads, j)
            assert (wo[j, P:] == 7.0).all(), "write past P"


def test_shape_tile_major_addressing():
    """Tile-major rows: coordinate p of row r sits at r*T + (p // T)*R*T + p % T."""
    from synth.device import ShapePass, ShapeRow
    dev = torch.device("cuda:0")
    T, R, P = 2048, 3, 2048 * 2 + 1024 + 8
    tiles = (P + T - 1) // T
    buf = torch.randn(tiles * R * T, device=dev)
    out = torch.full((tiles * R * T,), -1.0, device=dev)
    before = buf.clone()
    rows = [ShapeRow(buf, r * T, write=(r == 1)) for r in range(R)]
    ShapePass(rows + [ShapeRow(out, T, read=False)], P, tile=T,
              tile_stride=R * T * 4).launch()
    torch.cuda.synchronize()
    assert torch.equal(buf.view(torch.int32), before.view(torch.int32))
    p = np.arange(P)
    pos = lambda r: r * T + (p // T) * R * T + p % T  # noqa: E731
    host = buf.cpu()
    acc = np.zeros(P // 4, dtype=np.uint32)
    for r in range(R):
        acc ^= np.bitwise_xor.reduce(_words_f32(host[pos(r)]), axis=1)
    o = out.cpu()
    assert np.array_equal(_words_f32(o[pos(1)]), np.repeat(acc[:, None], 4, axis=1))
    untouched = np.ones(o.numel(), dtype=bool)
    untouched[pos(1)] = False
    assert (o[torch.from_numpy(untouched)] == -1.0).all()


def test_shape_pass_rejects_rows_that_do_not_fit():
    from synth.device import ShapePass, ShapeRow
    dev = torch.device("cuda:0")
    x = torch.zeros(1000, device=dev)
    with pytest.raises(ValueError):
        ShapePass([ShapeRow(x, 8)], 996)      # would reach element 1003
    with pytest.raises(ValueError):
        ShapePass([ShapeRow(x, 2)], 8)        # not 16-byte aligned
    with pytest.raises(ValueError):
        ShapePass([ShapeRow(x)], 10)          # P not a multiple of 4
    with pytest.raises(ValueError):           # tile layout past the buffer
        ShapePass([ShapeRow(x)], 1024 + 4, tile=1024, tile_stride=4096)
    ShapePass([ShapeRow(x, 4)], 996)          # exactly fits


def _fill_state(st, grads, seed):
    """Random bits in every row the synchronisation steps touch (finite
    values; the order kernel never looks at them) and a canary in the pads."""
    gen = torch.Generator(device="cpu").manual_seed(seed)
    for t in [st.params, st.mom, st.slow_mom, st.anchor, grads] + \
             ([st.mom2] if st.mom2 is not None else []):
        t.copy_(torch.randn(t.shape, generator=gen).to(t.dtype))
        if t.dim() == 2:
            t[:, st.P:] = 3.0


@pytest.mark.parametrize("method,adamw,W,pdt,gdt,mdt", [
    ("cpdp", False, 8, "f32", "f32", "f32"),
    ("cpdp", False, 4, "bf16", "f32", "f32"),
    ("cpdp", False, 8, "bf16", "bf16", "bf16"),
    ("cpdp", False, 16, "f32", "bf16", "f32"),
    ("cpdp", True, 8, "f32", "f32", "f32"),
    ("localsgd", False, 8, "f32", "f32", "f32"),
    ("localsgd", True, 4, "bf16", "f32", "f32"),
    ("ddp", False, 8, "f32", "f32", "f32"),
    ("ddp", True, 16, "bf16", "f32", "f32"),
])
def test_shape_sync_order_keeps_state_bits(method, adamw, W, pdt, gdt, mdt):
    """The library-order shape pass over a live state's rows: every row it
    writes back keeps its bits, the pads are untouched, and LocalSGD's
    write-only anchor gets the XOR of every row read."""
    import bench
    from paper_2607_21224_amd.state import CpdpState
    from synth.device import ShapeSyncPass
    P = 256 * 20 + 12  # twenty full 256-coordinate blocks and a partly used last one
    st = CpdpState(W, P, K=2, param_dt=pdt, grad_dt=gdt, mom_dt=mdt, adamw=adamw)
    grads = torch.empty((W, st.ld), device="cuda",
                        dtype=torch.bfloat16 if gdt == "bf16" else torch.float32)
    _fill_state(st, grads, seed=W * 7 + len(method))
    rows = bench.sync_shape_rows(st, grads, method, adamw)
    before = [r.tensor.clone() for r in rows]
    ShapeSyncPass(rows, P, method, adamw, W).launch()
    torch.cuda.synchronize()
    acc = np.zeros(P // 4, dtype=np.uint32)
    for r, b in zip(rows, before):
        if not r.read:
            continue
        view = torch.int16 if r.esize == 2 else torch.int32
        assert torch.equal(r.tensor.view(view), b.view(view)), (method, r.offset)
        seg = r.tensor.view(-1)[r.offset:r.offset + P]
        words = _words_bf16(seg) if r.esize == 2 else _words_f32(seg)
        acc ^= np.bitwise_xor.reduce(words, axis=1)
    if method == "localsgd":
        got = _words_f32(st.anchor[:P])
        assert np.array_equal(got, np.repeat(acc[:, None], 4, axis=1))


def test_shape_sync_pass_refuses_other_patterns():
    import bench
    from paper_2607_21224_amd.state import CpdpState
    from synth.device import ShapeRow, ShapeSyncPass
    st = CpdpState(8, 1024, K=2)
    grads = torch.zeros((8, st.ld), device="cuda")
    rows = bench.sync_shape_rows(st, grads, "cpdp", False)
    ShapeSyncPass(rows, 1024, "cpdp", False, 8)
    with pytest.raises(ValueError):
        ShapeSyncPass(rows, 1024, "ddp", False, 8)        # two rows too many
    with pytest.raises(ValueError):
        ShapeSyncPass(rows[::-1], 1024, "cpdp", False, 8)  # order
    with pytest.raises(ValueError):
        ShapeSyncPass(rows, 1024, "cpdp", True, 8)        # no second moments
    swapped = list(rows)
    swapped[0] = ShapeRow(st.mom, 0, write=True)          # a written row where g is read only
    with pytest.raises(ValueError):
        ShapeSyncPass(swapped, 1024, "cpdp", False, 8)
    st2 = CpdpState(2, 1024, K=2)
    with pytest.raises(ValueError):                       # W without an order kernel
        ShapeSyncPass(bench.sync_shape_rows(st2, grads[:2], "cpdp", False), 1024,
                      "cpdp", False, 2)
