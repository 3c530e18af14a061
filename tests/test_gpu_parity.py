"""GPU parity: libmsda (HIP, gfx950) against the CPU oracle, element by element.

Every case prints its name before it touches the GPU. Small cases cover many tiles, ragged
query tails, channel widths that exercise every lane layout (1..8 channels per lane, 1..64 lanes
per query, several channel chunks), many levels / points (several LDS phases), fp16 and fp32.
The full-size cases are the benchmark's workloads, compared on every output element.
"""
import numpy as np
import pytest

from paper_2505_14022_amd import msda, workloads
from gpu_util import check_parity, normwise, require_gpu, run_gpu, run_oracle, say, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    require_gpu()


SMALL = [
    # N, M, D, shapes, P, Lq, dtype
    (1, 2, 8, ((8, 8), (4, 4)), 2, 16, "f32"),
    (2, 3, 1, ((7, 5), (3, 2)), 3, 45, "f32"),
    (2, 3, 2, ((7, 5), (3, 2)), 3, 45, "f16"),
    (1, 4, 3, ((9, 13),), 4, 70, "f32"),
    (1, 4, 3, ((9, 13),), 4, 70, "f16"),
    (2, 2, 12, ((6, 10), (3, 5), (2, 2)), 2, 33, "f32"),
    (2, 2, 12, ((6, 10), (3, 5), (2, 2)), 2, 33, "f16"),
    (3, 8, 32, ((20, 30), (10, 15), (5, 8), (3, 4)), 4, 257, "f32"),
    (3, 8, 32, ((20, 30), (10, 15), (5, 8), (3, 4)), 4, 257, "f16"),
    (1, 1, 64, ((11, 7), (6, 4)), 8, 101, "f32"),
    (1, 2, 96, ((12, 9), (1, 1)), 3, 40, "f32"),
    (1, 2, 96, ((12, 9), (1, 1)), 3, 40, "f16"),
    (1, 2, 260, ((5, 6), (3, 3)), 2, 19, "f32"),   # two channel chunks per lane group
    (1, 2, 1032, ((4, 4),), 2, 9, "f16"),          # two channel chunks at fp16
    (2, 8, 32, ((16, 24), (8, 12), (4, 6), (2, 3)), 8, 150, "f32"),  # K = 32: two LDS phases
    (1, 2, 16, tuple((4 + l, 3 + 2 * l) for l in range(16)), 9, 50, "f32"),  # L = 16, K = 144
    (2, 3, 33, ((10, 10), (5, 5)), 3, 77, "f32"),
    (1, 1, 256, ((30, 40),), 1, 500, "f32"),
]


@pytest.mark.parametrize("path", ["owner", "atomic"])
@pytest.mark.parametrize("case", SMALL, ids=lambda c: f"N{c[0]}M{c[1]}D{c[2]}L{len(c[3])}P{c[4]}Lq{c[5]}{c[6]}")
def test_small_parity(case, path):
    N, M, D, shapes, P, Lq, dt = case
    inp = workloads.random_case(N, M, D, shapes, P, Lq, dt, seed=1000 + D + Lq)
    say(f"small case {inp.w.name} ({path} grad_value)")
    check_parity(inp, workspace="owner" if path == "owner" else None)


# As many queries as value pixels, each query at its own pixel (encoder self-attention): the forward
# and backward kernels deal the query chunks to the XCDs in bands of rows of every level. Row counts
# that do not divide by 8 leave bands of different sizes (workgroups past the end of a band exit);
# the first three grids are large enough that the backward does not split samples (which would use
# eighths of the query index instead); the last one is not.
BANDS = [
    ("detr_encoder", 2, ((40, 60), (20, 30), (10, 15), (5, 8))),
    ("swin5_f16", 2, ((66, 80), (33, 40), (17, 20), (9, 10), (5, 5))),
    ("bev_tsa_f16", 8, ((45, 37),)),
    # a small grid: the forward takes the bands, the backward splits samples and takes query eighths
    ("detr_encoder", 1, ((12, 10), (6, 5))),
]


@pytest.mark.parametrize("path", ["owner", "atomic"])
@pytest.mark.parametrize("case", BANDS, ids=lambda c: f"{c[0]}_N{c[1]}_S{sum(h * w for h, w in c[2])}")
def test_band_arrangement(case, path):
    base, N, shapes = case
    S = sum(h * w for h, w in shapes)
    w = workloads.scaled(workloads.BY_NAME[base], N=N, Lq=S, shapes=shapes, name=f"{base}_bands_N{N}_S{S}")
    say(f"bands of rows: {w.name} ({path} grad_value)")
    check_parity(workloads.generate(w), workspace="owner" if path == "owner" else None)


@pytest.mark.parametrize("seed", range(3))
def test_dense_coarse_levels_split_tiles(seed):
    # many queries on small maps: tiles see more samples than one work item folds, so tiles are
    # split and their rows are added with atomics
    inp = workloads.random_case(2, 4, 32, ((12, 10), (3, 5), (1, 2)), 8, 3000, "f32", seed=40 + seed,
                                lo=0.2, hi=0.6)
    say(f"split tiles seed {seed}")
    check_parity(inp, workspace="owner")


def test_many_tiles_multi_pass_scan():
    # 128 slabs x 525 tiles: the bin scan runs over more than 256 workgroups (the last one scans
    # their totals in several passes), and most of the scatter's workgroups only prepare work items
    inp = workloads.random_case(16, 8, 4, ((168, 200),), 2, 48, "f32", seed=77)
    say("many tiles: multi-pass scan of workgroup totals")
    check_parity(inp, workspace="owner")


def _hot_cell_case(n_hot: int, n_spread: int, seed: int):
    """One 8 x 8 map (one fold tile per slab, one work item): n_hot samples of each slab fall in one
    pixel cell (one key), the other n_spread are spread over the whole map."""
    P, Lq = 4, (n_hot + n_spread) // 4
    inp = workloads.random_case(1, 2, 32, ((8, 8),), P, Lq, "f32", seed=seed)
    rng = np.random.default_rng(seed)
    loc = inp.loc.reshape(1, Lq, 2, P, 2)
    for m in range(2):
        flat = loc[0, :, m].reshape(-1, 2)  # (q, p) order
        flat[:] = rng.uniform(0.02, 0.98, size=flat.shape).astype(np.float32)
        hot = rng.choice(flat.shape[0], size=n_hot, replace=False)
        # h_im in (3.1, 3.9), w_im in (4.1, 4.9): the cell whose top-left corner is pixel (3, 4)
        flat[hot, 0] = ((rng.uniform(4.1, 4.9, size=n_hot) + 0.5) / 8).astype(np.float32)
        flat[hot, 1] = ((rng.uniform(3.1, 3.9, size=n_hot) + 0.5) / 8).astype(np.float32)
        loc[0, :, m] = flat.reshape(Lq, P, 2)
    return inp


@pytest.mark.parametrize("n_hot,n_spread", [(200, 300), (352, 148), (480, 20)])
def test_fold_hot_key(n_hot, n_spread):
    # (200, 300) and (352, 148): runs average under 12 records, so the item is summed by work units,
    # and the hot key's 25 or 44 pieces fill whole rounds that add in up to 16 passes by rank;
    # (480, 20): the slice walk, with most slices ending on the hot key
    inp = _hot_cell_case(n_hot, n_spread, seed=900 + n_hot)
    say(f"fold hot key: {n_hot} samples in one cell, {n_spread} spread")
    check_parity(inp, workspace="owner")


@pytest.mark.parametrize("lo,hi", [(-0.6, 1.6), (0.0, 1.0), (0.45, 0.55)])
def test_location_ranges(lo, hi):
    inp = workloads.random_case(2, 4, 32, ((13, 17), (7, 9)), 4, 123, "f32", seed=7, lo=lo, hi=hi)
    say(f"location range [{lo}, {hi}]")
    check_parity(inp, workspace="owner")


@pytest.mark.parametrize("w", workloads.WORKLOADS, ids=lambda w: w.name)
def test_workload_full_size(w):
    say(f"full-size workload {w.name}: N={w.N} M={w.M} D={w.D} S={w.S} Lq={w.Lq} L={w.L} P={w.P} {w.dtype}")
    inp = workloads.generate(w)
    check_parity(inp)


@pytest.mark.parametrize("name", ["tiny", "detr_decoder"])
def test_sparse_workloads_owner_path(name):
    # these take the atomic path by default; the owner-computes path must agree as well
    w = workloads.BY_NAME[name]
    say(f"full-size workload {w.name} with owner-computes grad_value")
    check_parity(workloads.generate(w), workspace="owner")


def test_workload_full_size_atomic_path():
    w = workloads.BY_NAME["detr_encoder"]
    say(f"full-size workload {w.name} with atomic grad_value")
    check_parity(workloads.generate(w), workspace=None)


def test_pixel_centres_are_exact():
    # power-of-two maps: pixel-centre locations give h_im, w_im exactly integral -> a plain gather
    import torch

    rng = np.random.default_rng(5)
    shapes = ((16, 8), (8, 4), (4, 2))
    inp = workloads.random_case(2, 4, 32, shapes, 2, 64, "f32", seed=5)
    for l, (H, W) in enumerate(shapes):
        h = rng.integers(0, H, size=inp.loc.shape[:3] + (inp.loc.shape[4],))
        w = rng.integers(0, W, size=h.shape)
        inp.loc[:, :, :, l, :, 0] = (w + 0.5) / W
        inp.loc[:, :, :, l, :, 1] = (h + 0.5) / H
    say("pixel-centre gather")
    gpu = run_gpu(inp)
    ref = run_oracle(inp)
    # one corner of weight 1 per sample: the only rounding is the weighted sum over samples
    assert normwise(gpu["out"], ref["out"]) < 1e-6
    check_parity(inp, gpu=gpu, ref=ref)


def test_off_map_samples_contribute_nothing():
    inp = workloads.random_case(1, 2, 32, ((6, 9), (3, 4)), 2, 40, "f32", seed=6)
    inp.loc[..., 0] = -0.6  # w_im <= -1 on every level: every sample off the map
    say("off-map samples")
    gpu = run_gpu(inp)
    assert np.all(gpu["out"] == 0) and np.all(gpu["grad_value"] == 0)
    assert np.all(gpu["grad_loc"] == 0) and np.all(gpu["grad_attn"] == 0)


def test_empty_problems():
    import torch

    say("empty problems (Lq = 0 zeroes grad_value, N = 0 is a no-op)")
    inp = workloads.random_case(2, 2, 8, ((4, 4),), 2, 0, "f32", seed=8)
    d = to_device(inp)
    gv = torch.full(tuple(inp.value.shape), 7.0, device="cuda")
    out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn)
    msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, grad_value=gv)
    torch.cuda.synchronize()
    assert out.shape == (2, 0, 16)
    assert torch.all(gv == 0).item()
    inp = workloads.random_case(0, 2, 8, ((4, 4),), 2, 5, "f32", seed=8)
    d = to_device(inp)
    out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn)
    msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out)
    torch.cuda.synchronize()


def test_outputs_fully_overwritten_and_deterministic():
    import torch

    inp = workloads.random_case(2, 8, 32, ((20, 30), (10, 15)), 4, 300, "f32", seed=9)
    d = to_device(inp)
    say("overwrite + determinism")
    outs = []
    for fill in (float("nan"), 3.0):
        out = torch.full((2, 300, 256), fill, device="cuda")
        gv = torch.full(tuple(inp.value.shape), fill, device="cuda")
        gl = torch.full(tuple(inp.loc.shape), fill, device="cuda")
        ga = torch.full(tuple(inp.attn.shape), fill, device="cuda")
        msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn, out=out)
        msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, gv, gl, ga)
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (out, gv, gl, ga)])
    a, b = outs
    assert np.array_equal(a[0], b[0]), "forward is not bitwise reproducible"
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3]), "grad_loc / grad_attn not reproducible"
    assert np.all(np.isfinite(a[1])) and normwise(a[1], b[1]) < 1e-6


def test_side_stream():
    import torch

    inp = workloads.random_case(1, 4, 32, ((12, 10), (6, 5)), 4, 200, "f32", seed=10)
    d = to_device(inp)
    say("side stream")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn, stream=s)
        gv, gl, ga = msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, stream=s)
    s.synchronize()
    ref = run_oracle(inp)
    assert normwise(out.cpu().numpy(), ref["out"]) <= 1e-5
    assert normwise(gv.cpu().numpy(), ref["grad_value"]) <= 1e-4


def test_backward_on_two_user_streams():
    # the owner-computes backward forks its grad_value work onto a library stream and joins it
    # back; calls on two user streams from one thread must each see their own inputs
    import torch

    cases = [workloads.random_case(1, 4, 32, ((24, 20), (12, 10)), 4, 2000, "f32", seed=20 + i) for i in range(2)]
    say("backward on two user streams")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    dev = [to_device(c) for c in cases]
    torch.cuda.synchronize()
    res = []
    for c, d, st in zip(cases, dev, streams):
        with torch.cuda.stream(st):
            res.append(msda.backward(d.value, c.shapes, c.starts, d.loc, d.attn, d.grad_out, workspace="owner",
                                     stream=st))
    torch.cuda.synchronize()
    for c, r in zip(cases, res):
        ref = run_oracle(c)
        assert normwise(r[0].cpu().numpy(), ref["grad_value"]) <= 1e-4
        assert normwise(r[1].cpu().numpy(), ref["grad_loc"]) <= 1e-3
        assert normwise(r[2].cpu().numpy(), ref["grad_attn"]) <= 1e-3


def test_backward_graph_replays():
    # forward + backward captured into a graph (the grad_value fork and join included), replayed
    # several times with eager work in between; every replay must match the eager results
    import torch

    inp = workloads.random_case(2, 4, 32, ((24, 20), (12, 10)), 4, 1500, "f32", seed=31)
    d = to_device(inp)
    say("graph capture and replays of forward + backward")
    w = inp.w
    ws = torch.empty(msda.workspace_size(inp.shapes, inp.starts, w.N, w.S, w.M, w.D, w.Lq, w.L, w.P, msda.MSDA_F32,
                                         msda.MSDA_WORKSPACE_OWNER),
                     dtype=torch.uint8, device="cuda")
    out = torch.empty((2, 1500, 128), device="cuda")
    gv = torch.empty(tuple(inp.value.shape), device="cuda")
    gl = torch.empty(tuple(inp.loc.shape), device="cuda")
    ga = torch.empty(tuple(inp.attn.shape), device="cuda")

    def step(stream):
        msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn, out=out, stream=stream)
        msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, gv, gl, ga, workspace=ws,
                      stream=stream)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    eager = [x.cpu().numpy() for x in (out, gv, gl, ga)]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step(s)
    torch.cuda.synchronize()
    for rep in range(3):
        for x in (out, gv, gl, ga):
            x.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [x.cpu().numpy() for x in (out, gv, gl, ga)]
        assert np.array_equal(got[0], eager[0]), f"replay {rep}: out differs"
        assert np.array_equal(got[2], eager[2]) and np.array_equal(got[3], eager[3]), f"replay {rep}: grad_loc/attn"
        assert np.all(np.isfinite(got[1])) and normwise(got[1], eager[1]) < 1e-6, f"replay {rep}: grad_value"
        step(torch.cuda.current_stream())  # eager work between the replays
        torch.cuda.synchronize()


def test_adjoint_identities_on_gpu_results():
    # out is linear in value and attn: <g, out> = <grad_value, value> = <grad_attn, attn>
    w = workloads.BY_NAME["detr_encoder"]
    inp = workloads.generate(w)
    say("adjoint identities at the DETR-encoder shape")
    gpu = run_gpu(inp)
    lhs = float(np.sum(inp.grad_out.astype(np.float64) * gpu["out"].astype(np.float64)))
    r1 = float(np.sum(gpu["grad_value"].astype(np.float64) * inp.value.astype(np.float64)))
    r2 = float(np.sum(gpu["grad_attn"].astype(np.float64) * inp.attn.astype(np.float64)))
    scale = float(np.sum(np.abs(inp.grad_out.astype(np.float64) * gpu["out"])))
    assert abs(lhs - r1) <= 1e-5 * scale and abs(lhs - r2) <= 1e-5 * scale


def _segment_stream(torch, ptr):
    for seg in torch.cuda.memory_snapshot():
        if seg["address"] <= ptr < seg["address"] + seg["total_size"]:
            return seg["stream"]
    return None


def test_binding_allocates_on_the_call_stream():
    # outputs and workspaces the binding allocates belong to the stream the kernels run on, so the
    # caching allocator cannot hand them to other work while the call is still running there
    import torch

    inp = workloads.random_case(1, 4, 32, ((24, 20), (12, 10)), 4, 2000, "f32", seed=41)
    d = to_device(inp)
    say("binding allocations on a stream other than the current one")
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    assert torch.cuda.current_stream() != s
    out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn, stream=s)
    gv, gl, ga = msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, workspace="owner",
                               stream=s)
    for t in (out, gv, gl, ga):
        assert _segment_stream(torch, t.data_ptr()) == s.cuda_stream
    # memory allocated and written on the current stream right away does not disturb the call
    junk = [torch.full((1 << 22,), float("nan"), device="cuda") for _ in range(4)]
    s.synchronize()
    torch.cuda.synchronize()
    del junk
    check_parity(inp, gpu={"out": out.cpu().numpy(), "grad_value": gv.cpu().numpy(),
                           "grad_loc": gl.cpu().numpy(), "grad_attn": ga.cpu().numpy()})


def test_release_and_recreate_side_streams():
    inp = workloads.random_case(1, 4, 32, ((24, 20), (12, 10)), 4, 2000, "f32", seed=42)
    say("msda_release between backward calls")
    a = run_gpu(inp, workspace="owner")
    msda.release()
    b = run_gpu(inp, workspace="owner")  # the side stream is created again
    msda.release()
    msda.release()  # nothing left to release
    ref = run_oracle(inp)
    for g in (a, b):
        check_parity(inp, gpu=g, ref=ref)


@pytest.mark.parametrize("name", ["tiny", "detr_decoder", "detr_encoder"])
def test_atomic_entry_zeroes_then_adds(name):
    # msda_backward_atomic zeroes grad_value and then adds every corner contribution with fp32
    # atomics on the same stream: outputs prefilled with NaN show any element that was not zeroed
    # first or not written, and a stream other than the current one checks the stream handling
    import torch

    w = workloads.BY_NAME[name]
    inp = workloads.generate(w)
    d = to_device(inp)
    say(f"atomic entry point on NaN-filled outputs, side stream: {name}")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        gv = torch.full(tuple(inp.value.shape), float("nan"), device="cuda")
        gl = torch.full(tuple(inp.loc.shape), float("nan"), device="cuda")
        ga = torch.full(tuple(inp.attn.shape), float("nan"), device="cuda")
    out = msda.forward(d.value, inp.shapes, inp.starts, d.loc, d.attn, stream=s)
    msda.backward(d.value, inp.shapes, inp.starts, d.loc, d.attn, d.grad_out, gv, gl, ga, workspace=None, stream=s)
    s.synchronize()
    gpu = {"out": out.cpu().numpy(), "grad_value": gv.cpu().numpy(), "grad_loc": gl.cpu().numpy(),
           "grad_attn": ga.cpu().numpy()}
    check_parity(inp, gpu=gpu, entry="atomic")
