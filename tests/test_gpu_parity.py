"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Tolerances: fp32 workloads 1e-4 relative against the float64 oracle
(norm-wise per tensor, plain relative on each loss).  bf16 workloads 2e-2
relative against the oracle that rounds to bf16 the tensors the GPU stores in
bf16, and against the float64 oracle within 2e-2 on losses and parameters and
within what bf16 arithmetic itself attains on gradients and moments (see
tests/gpu_util.check_bf16).  All schedules (serial, overlapped, and both
captured as HIP graphs) must agree bit for bit.
"""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_18469_amd import erase, synth
from tests.gpu_util import (assert_bit_identical, check_bf16, check_f32, compare, run_gpu, run_gpu_nosync,
                            run_oracle)

pytestmark = pytest.mark.gpu

SCHEDS = ["serial", "overlap", "serial_graph", "overlap_graph", "pipeline", "overlap_adam_end"]


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _mixed_fp32(batch=150):
    blocks = [
        {"input": "x", "layers": [("cross", 100, 100), ("cross", 100, 100), ("linear_relu", 100, 70),
                                  ("linear_relu", 70, 50)], "lam": 1.0},
        {"input": "prev", "layers": [("linear_relu", 50, 90), ("linear_relu", 90, 33)], "lam": 0.5},
        {"input": "x", "layers": [("linear_relu", 100, 130)], "lam": 2.0},
    ]
    return synth.custom("f32", batch, 100, blocks, label_p=0.3)


def test_tiny_fp32_three_steps_vs_oracle():
    _say("case: tiny fp32 3 steps")
    cfg = synth.config("tiny")
    params, batches = synth.make_workload(cfg, 0, 3)
    _, g = run_gpu(cfg, params, batches, "overlap")
    r = run_oracle(cfg, params, batches)
    compare(cfg, g, r, 1e-4)


def test_tiny_chain_fp32_vs_oracle():
    _say("case: tiny_chain fp32 3 steps")
    cfg = synth.config("tiny_chain")
    params, batches = synth.make_workload(cfg, 1, 3)
    _, g = run_gpu(cfg, params, batches, "overlap")
    r = run_oracle(cfg, params, batches)
    compare(cfg, g, r, 1e-4)


@pytest.mark.parametrize("batch", [150, 1, 64, 257])
def test_cross_chain_mixed_fp32_vs_oracle(batch):
    """Cross layers, a chained block and ragged shapes spanning several 64x64
    tiles, fp32."""
    _say(f"case: mixed fp32 batch={batch}")
    cfg = _mixed_fp32(batch)
    params, batches = synth.make_workload(cfg, 2, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    r = run_oracle(cfg, params, batches)
    compare(cfg, g, r, 1e-4)


def test_odd_small_dims_fp32():
    _say("case: odd small dims fp32")
    blocks = [{"input": "x", "layers": [("linear_relu", 3, 1)], "lam": 1.0},
              {"input": "prev", "layers": [("linear_relu", 1, 5), ("linear_relu", 5, 2)], "lam": 1.0}]
    cfg = synth.custom("f32", 7, 3, blocks, label_p=0.5)
    params, batches = synth.make_workload(cfg, 4, 2)
    _, g = run_gpu(cfg, params, batches)
    r = run_oracle(cfg, params, batches)
    compare(cfg, g, r, 1e-4)


@pytest.mark.parametrize("name", ["tiny", "tiny_chain"])
def test_schedules_bit_identical_fp32(name):
    _say(f"case: schedules bit-identical {name}")
    cfg = synth.config(name)
    params, batches = synth.make_workload(cfg, 0, 3)
    runs = [run_gpu(cfg, params, batches, s)[1] for s in SCHEDS]
    for other in runs[1:]:
        assert_bit_identical(runs[0], other)


def _ctr_small(batch=1000, blocks=2):
    cfg = synth.config("ctr_mlp", batch=batch, ctr_rows=5000)
    cfg["blocks"] = cfg["blocks"][:blocks]
    return cfg


@pytest.mark.parametrize("batch", [1000, 777])
def test_ctr_mlp_bf16_small_vs_oracle(batch):
    """Full CTR widths (1677->512->256->128), 2 blocks, ragged batches; 777
    pads to an odd number of k-steps in the weight-gradient GEMMs."""
    _say(f"case: ctr_mlp bf16 batch={batch}")
    cfg = _ctr_small(batch=batch)
    params, batches = synth.make_workload(cfg, 0, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    _say("  ", check_bf16(cfg, g, params, batches))


def _mixed_bf16(batch):
    # last layers of 64, 128 (head fused into the forward GEMM; the first is
    # read by a chained block), 40 on a single-layer block (no input gradient
    # of the last layer) and 200 (standalone head kernel)
    blocks = [
        {"input": "x", "layers": [("linear_relu", 200, 96), ("linear_relu", 96, 64)], "lam": 1.0},
        {"input": "prev", "layers": [("linear_relu", 64, 100), ("linear_relu", 100, 128)], "lam": 0.5},
        {"input": "x", "layers": [("linear_relu", 200, 40)], "lam": 2.0},
        {"input": "x", "layers": [("linear_relu", 200, 72), ("linear_relu", 72, 200)], "lam": 1.0},
    ]
    return synth.custom("bf16", batch, 200, blocks, label_p=0.3)


@pytest.mark.parametrize("batch", [333, 64])
def test_fused_and_standalone_head_bf16_vs_oracle(batch):
    """bf16 blocks whose head is fused into the last forward GEMM (chained and
    not, with and without an input gradient of the last layer) next to one
    with the standalone head kernel; every schedule gives the same bits."""
    _say(f"case: mixed bf16 heads batch={batch}")
    cfg = _mixed_bf16(batch)
    params, batches = synth.make_workload(cfg, 6, 2)
    runs = [run_gpu(cfg, params, batches, s)[1] for s in SCHEDS]
    for other in runs[1:]:
        assert_bit_identical(runs[0], other)
    _say("  ", check_bf16(cfg, runs[0], params, batches))
    tr = erase.Trainer(cfg, params)
    tr.set_timing(True)
    tr.step(*tr.device_batch(*batches[0]), "serial")
    tr.sync()
    kinds = [(r["block"], r["kind"]) for r in tr.read_timing()[1:]]
    assert [b for b, k in kinds if k == "fwd_head_gemm"] == [0, 1, 2]
    assert [b for b, k in kinds if k == "head_bce"] == [3]
    tr.close()


@pytest.mark.parametrize("name", ["tiny_chain", "mixed", "odd"])
def test_undetached_fp32_vs_oracle(name):
    """The conventional (undetached) baseline: gradients cross the cuts of a
    chain; fp32 against the float64 oracle's undetached step."""
    _say(f"case: undetached fp32 {name}")
    if name == "tiny_chain":
        cfg = synth.config("tiny_chain")
    elif name == "mixed":
        cfg = _mixed_fp32(150)
    else:
        blocks = [{"input": "x", "layers": [("linear_relu", 3, 1)], "lam": 1.0},
                  {"input": "prev", "layers": [("linear_relu", 1, 5), ("linear_relu", 5, 2)], "lam": 1.0}]
        cfg = synth.custom("f32", 7, 3, blocks, label_p=0.5)
    params, batches = synth.make_workload(cfg, 8, 3)
    _, g = run_gpu(cfg, params, batches, "undetached")
    r = run_oracle(cfg, params, batches, detach=False)
    compare(cfg, g, r, 1e-4)
    if name != "odd":  # (the odd case's 1-wide cut is a dead ReLU on this batch: nothing flows back)
        # and it is not the detached step
        rd = run_oracle(cfg, params, batches)
        assert max(float(np.abs(a - b).max()) for a, b in zip(g[0]["grads"][0], rd[0]["grads"][0])) > 1e-6


def test_undetached_bf16_chain_vs_oracle():
    _say("case: undetached bf16 deep chain")
    cfg = synth.config("deep_chain", batch=384)
    cfg["blocks"] = cfg["blocks"][:5]
    params, batches = synth.make_workload(cfg, 9, 2)
    _, g = run_gpu(cfg, params, batches, "undetached")
    _say("  ", check_bf16(cfg, g, params, batches, detach=False))


def _replayed(cfg, params, batches, schedule, steps):
    """`steps` steps cycling over the same device batches (a graph schedule
    replays its graph from the third step on), the state read back after each."""
    tr = erase.Trainer(cfg, params, keep_grads=True)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    recs = []
    for i in range(steps):
        xd, yd = dev[i % len(dev)]
        tr.step(xd, yd, schedule)
        tr.sync()
        p, m, v, g = tr.flat_state()
        recs.append({"losses": tr.losses.cpu().numpy().copy(), "params": p, "m": m, "v": v, "grads": g})
    tr.close()
    return recs


@pytest.mark.parametrize("name", ["tiny_chain", "deep_chain5"])
def test_undetached_graph_replays_match_eager(name):
    """The conventional step captured as a HIP graph: every replay, with host
    reads in between, bit-identical to the eager conventional step."""
    _say(f"case: undetached_graph {name}")
    if name == "tiny_chain":
        cfg = synth.config("tiny_chain")
    else:
        cfg = synth.config("deep_chain", batch=256)
        cfg["blocks"] = cfg["blocks"][:5]
    params, batches = synth.make_workload(cfg, 11, 2)
    assert_bit_identical(_replayed(cfg, params, batches, "undetached", 5),
                         _replayed(cfg, params, batches, "undetached_graph", 5))


def test_undetached_equals_serial_on_shared_input_and_rejects_cross_chains():
    _say("case: undetached on shared input; unsupported chain")
    cfg = _ctr_small(batch=300, blocks=2)
    params, batches = synth.make_workload(cfg, 4, 2)
    assert_bit_identical(run_gpu(cfg, params, batches, "serial")[1], run_gpu(cfg, params, batches, "undetached")[1])
    blocks = [{"input": "x", "layers": [("linear_relu", 8, 6)], "lam": 1.0},
              {"input": "prev", "layers": [("cross", 6, 6), ("linear_relu", 6, 4)], "lam": 1.0}]
    bad = synth.custom("f32", 16, 8, blocks)
    p2, b2 = synth.make_workload(bad, 0, 1)
    tr = erase.Trainer(bad, p2)
    x, y = tr.device_batch(*b2[0])
    with pytest.raises(erase.EraseError):
        tr.step(x, y, "undetached")
    tr.step(x, y, "serial")  # the context stays usable
    tr.sync()
    tr.close()


def test_ctr_mlp_bf16_schedules_bit_identical():
    """Serial, overlapped and graph schedules, with 1 and 3 backward streams,
    produce the same bits."""
    _say("case: ctr_mlp bf16 schedules bit-identical")
    cfg = _ctr_small(batch=777, blocks=4)
    params, batches = synth.make_workload(cfg, 3, 2)
    runs = [run_gpu(cfg, params, batches, s)[1] for s in SCHEDS]
    runs += [run_gpu(cfg, params, batches, s, bwd_streams=3)[1] for s in ("overlap", "overlap_graph")]
    for other in runs[1:]:
        assert_bit_identical(runs[0], other)


@pytest.mark.parametrize("name,streams", [("ctr_small", 2), ("deep_chain", 3), ("mixed", 1)])
def test_pipelined_steps_match_serial(name, streams):
    """PIPELINE steps enqueued back to back (no end-of-step join, so one
    step's last backwards overlap the next step's first forwards), and a mix
    of schedules, give the same bits as serial steps."""
    _say(f"case: pipelined steps, {name}, {streams} backward streams")
    if name == "ctr_small":
        cfg = _ctr_small(batch=640, blocks=4)
    elif name == "deep_chain":
        cfg = synth.config("deep_chain", batch=384)
    else:
        cfg = _mixed_fp32(200)
    params, batches = synth.make_workload(cfg, 11, 5)
    ref_l, ref = run_gpu_nosync(cfg, params, batches, ["serial"])
    got_l, got = run_gpu_nosync(cfg, params, batches, ["pipeline"], bwd_streams=streams)
    assert np.array_equal(ref_l.view(np.uint32), got_l.view(np.uint32))
    assert_bit_identical([ref], [got])
    mix_l, mix = run_gpu_nosync(cfg, params, batches, ["pipeline", "serial", "pipeline", "overlap_graph", "pipeline"],
                                bwd_streams=streams)
    assert np.array_equal(ref_l.view(np.uint32), mix_l.view(np.uint32))
    assert_bit_identical([ref], [mix])


@pytest.mark.parametrize("name,streams", [("ctr_small", 2), ("deep_chain", 2), ("deep_chain", 1), ("mixed", 3)])
def test_worker_dispatch_matches_serial(name, streams):
    """The backward streams' work enqueued by the library's worker thread
    (non-blocking dispatch): PIPELINE and OVERLAP steps back to back, and a
    mix with graph, serial and undetached-free schedules, give the same bits
    as serial steps dispatched from the caller."""
    _say(f"case: worker dispatch, {name}, {streams} backward streams")
    if name == "ctr_small":
        cfg = _ctr_small(batch=640, blocks=4)
    elif name == "deep_chain":
        cfg = synth.config("deep_chain", batch=384)
    else:
        cfg = _mixed_fp32(200)
    params, batches = synth.make_workload(cfg, 13, 6)
    ref_l, ref = run_gpu_nosync(cfg, params, batches, ["serial"])
    for scheds in (["pipeline"], ["overlap"], ["overlap_adam_end", "pipeline"],
                   ["pipeline", "pipeline", "serial", "overlap_graph", "pipeline", "overlap"]):
        got_l, got = run_gpu_nosync(cfg, params, batches, scheds, bwd_streams=streams, dispatch="worker")
        assert np.array_equal(ref_l.view(np.uint32), got_l.view(np.uint32)), scheds
        assert_bit_identical([ref], [got])


def test_worker_dispatch_switch_and_state_calls():
    """Switching dispatch modes between steps, and the state calls
    (step counter, timing) in the middle of worker-dispatched steps."""
    _say("case: worker dispatch switching")
    cfg = _ctr_small(batch=320, blocks=3)
    params, batches = synth.make_workload(cfg, 17, 6)
    ref_l, ref = run_gpu_nosync(cfg, params, batches, ["serial"])
    tr = erase.Trainer(cfg, params, keep_grads=True, bwd_streams=2)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    import torch
    outs = [torch.zeros(len(cfg["blocks"]), dtype=torch.float32, device="cuda") for _ in batches]
    modes = ["worker", "worker", "caller", "worker", "caller", "worker"]
    for i, (xd, yd) in enumerate(dev):
        tr.set_dispatch(modes[i])
        tr.step(xd, yd, "pipeline", losses=outs[i], wait_current=(i == 0))
        if i == 2:
            assert tr.get_step() == 3
        if i == 3:
            tr.set_timing(True)
            tr.set_timing(False)
    tr.sync()
    p, m, v, g = tr.flat_state()
    tr.close()
    got_l = np.stack([o.cpu().numpy() for o in outs])
    assert np.array_equal(ref_l.view(np.uint32), got_l.view(np.uint32))
    assert_bit_identical([ref], [{"losses": got_l[-1], "params": p, "m": m, "v": v, "grads": g}])
    tr2 = erase.Trainer(cfg, params)
    assert erase.lib().erase_set_dispatch(tr2.ctx, 5) == erase.ERR_INVALID_ARG
    tr2.close()


def test_caller_owned_streams():
    """Streams supplied by the caller (here torch streams) instead of the
    binding's own: same bits as the default construction."""
    import torch
    _say("case: caller-owned streams")
    cfg = _ctr_small(batch=256, blocks=3)
    params, batches = synth.make_workload(cfg, 21, 3)
    ref = run_gpu(cfg, params, batches, "overlap", bwd_streams=2)[1]
    streams = (torch.cuda.Stream(), [torch.cuda.Stream(), torch.cuda.Stream()])
    tr = erase.Trainer(cfg, params, keep_grads=True, streams=streams)
    assert tr.sf is streams[0] and tr.sbs == streams[1]
    got = run_gpu(cfg, params, batches, "overlap", trainer=tr)[1]
    tr.close()
    assert_bit_identical(ref, got)


def _bags(seed, M, T, rows, dim, n_dense, max_len, allow_empty=True):
    rng = np.random.Generator(np.random.PCG64(seed))
    tables = rng.normal(0, 1, size=(T, rows, dim)).astype(np.float32)
    dense = rng.lognormal(0, 1, size=(M, n_dense)).astype(np.float32)
    offsets = np.zeros((T, M + 1), dtype=np.int64)
    ids, base = [], 0
    for t in range(T):
        lens = rng.integers(0 if allow_empty else 1, max_len + 1, size=M)
        offsets[t, 0] = base
        offsets[t, 1:] = base + np.cumsum(lens)
        ids.append(rng.integers(0, rows, size=int(lens.sum())).astype(np.int32))
        base += int(lens.sum())
    return dense, offsets, np.concatenate(ids), tables


def _run_bags(dense, offsets, indices, tables, dtype, x_ld):
    import torch
    M = offsets.shape[1] - 1
    dev = "cuda"
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.full((M, x_ld), float("nan"), dtype=tdt, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    d = torch.from_numpy(dense).to(dev) if dense.shape[1] else None
    erase.embed_bags(d, torch.from_numpy(offsets).to(dev), torch.from_numpy(indices).to(dev),
                     torch.from_numpy(tables).to(dev), x, status)
    torch.cuda.synchronize()
    return x.float().cpu().numpy(), int(status.item())


@pytest.mark.parametrize("dtype,dim,n_dense,M,T", [("f32", 64, 13, 37, 5), ("bf16", 64, 13, 37, 5),
                                                   ("f32", 4, 0, 5, 3), ("bf16", 12, 3, 64, 2),
                                                   ("f32", 256, 1, 9, 2), ("bf16", 64, 13, 1, 26)])
def test_embed_bags_vs_oracle(dtype, dim, n_dense, M, T):
    """The embedding-bag input stage against the float64 oracle: ragged batch,
    empty bags, widths that leave lanes idle, no dense features."""
    _say(f"case: embed_bags {dtype} dim={dim} n_dense={n_dense} M={M} T={T}")
    dense, offsets, indices, tables = _bags(M * 31 + dim, M, T, 300, dim, n_dense, 7)
    width = n_dense + T * dim
    x_ld = (width + 5 + 7) // 8 * 8
    x, status = _run_bags(dense, offsets, indices, tables, dtype, x_ld)
    ref = oracle.embed_bags(dense.astype(np.float64), offsets, indices, tables.astype(np.float64))
    assert status == 0
    assert np.array_equal(x[:, width:], np.zeros((M, x_ld - width)))
    if dtype == "f32":
        # fp32 sum of <= 7 N(0,1) rows and fp32 log1p: a few ulp of the sum of magnitudes
        mag = oracle.embed_bags(dense.astype(np.float64), offsets, indices, np.abs(tables.astype(np.float64)))
        assert np.all(np.abs(x[:, :width] - ref) <= 4e-7 * (np.abs(mag) + 1e-30) * 8 + 1e-7 * np.abs(ref))
    else:
        # one bf16 rounding of an fp32 value: half an ulp (2^-9 relative) plus the fp32 error
        assert np.all(np.abs(x[:, :width] - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-6)


def test_embed_bags_full_ctr_shape():
    """The CTR workload's input stage at full size (4096 rows, 26 tables of
    100000 x 64, bags of 1..20 Zipf(1.1) ids): float32 output, pooled
    columns bit-identical to the input generator's float32 pooling in index
    order, and the float64 oracle within float32 rounding."""
    import torch
    _say("case: embed_bags full CTR shape")
    rng = np.random.Generator(np.random.PCG64(0))
    tabs = synth.CtrTables(rng)
    state = rng.bit_generator.state
    raw = synth.make_ctr_raw(tabs, 4096, rng)
    rng.bit_generator.state = state
    xg = synth.make_ctr_x(tabs, 4096, rng)
    tables = np.stack(tabs.tables)
    dense = raw["dense"].astype(np.float32)
    x, status = _run_bags(dense, raw["offsets"], raw["indices"], tables, "f32", 1680)
    assert status == 0
    assert np.array_equal(x[:, 13:1677].view(np.uint32), xg[:, 13:].view(np.uint32))
    assert np.array_equal(x[:, 1677:], np.zeros((4096, 3)))
    ref = oracle.embed_bags(dense.astype(np.float64), raw["offsets"], raw["indices"], tables.astype(np.float64))
    np.testing.assert_allclose(x[:, :1677], ref, rtol=1e-6, atol=2e-8)


def test_embed_bags_invalid_entries_flagged():
    """Out-of-range ids and reversed or out-of-range bag bounds read nothing:
    they contribute zero and set the status word; every other bag is exact."""
    _say("case: embed_bags invalid entries")
    dense, offsets, indices, tables = _bags(41, 16, 3, 50, 64, 2, 5, allow_empty=False)
    good_x, st = _run_bags(dense, offsets, indices, tables, "f32", 200)
    assert st == 0
    bad_idx = indices.copy()
    o = offsets
    bad_idx[o[1, 3]] = 50          # table 1, bag 3: first id past the last row
    bad_idx[o[2, 7]] = -1          # table 2, bag 7: negative id
    bad_off = offsets.copy()
    bad_off[0, 5] = bad_off[0, 6] + 1  # table 0: bag 4 runs past its end, bag 5 is reversed
    x, st = _run_bags(dense, bad_off, bad_idx, tables, "f32", 200)
    assert st == 1
    ref = oracle.embed_bags(dense.astype(np.float64), offsets, indices, tables.astype(np.float64))
    tab64 = tables.astype(np.float64)
    exp = ref.copy()
    exp[3, 2 + 64: 2 + 128] -= tab64[1][indices[o[1, 3]]]
    exp[7, 2 + 128: 2 + 192] -= tab64[2][indices[o[2, 7]]]
    # bag (0, 4) now reads indices[o[0,4] : o[0,6]+1] (valid range, longer); bag (0, 5) is reversed: zero
    exp[4, 2:66] = tab64[0][indices[o[0, 4]: o[0, 6] + 1]].sum(axis=0)
    exp[5, 2:66] = 0.0
    np.testing.assert_allclose(x[:, :194], exp, rtol=1e-5, atol=1e-5)
    for m in range(16):
        if m not in (3, 4, 5, 7):
            assert np.array_equal(x[m, :194], good_x[m, :194])


def _run_bags_bwd(offsets, indices, dx, n_dense, rows, dim, dtype):
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = torch.full((offsets.shape[0], rows, dim), float("nan"), dtype=torch.float32, device="cuda")
    erase.embed_bags_backward(torch.from_numpy(offsets).cuda(), torch.from_numpy(indices).cuda(),
                              torch.from_numpy(dx).cuda().to(tdt), n_dense, rows, dim, table_grad=g, status=status)
    torch.cuda.synchronize()
    return g.cpu().numpy(), int(status.item())


@pytest.mark.parametrize("dtype,dim,n_dense,M,T,rows,max_len", [("f32", 64, 13, 37, 5, 40, 7), ("bf16", 64, 13, 37, 5, 40, 7),
                                                                ("f32", 4, 0, 5, 3, 9, 3), ("f32", 256, 1, 9, 2, 300, 7),
                                                                ("bf16", 12, 3, 64, 2, 5, 90),
                                                                ("f32", 8, 0, 400, 1, 1, 90),
                                                                ("f32", 8, 0, 30000, 1, 30, 20),
                                                                ("bf16", 8, 0, 30000, 1, 500, 20)])
def test_embed_bags_backward_vs_oracle(dtype, dim, n_dense, M, T, rows, max_len):
    """Table gradients against the float64 oracle: empty bags, rows selected
    by no bag (zero), and with 5 rows and bags of up to 90 ids, rows selected
    by well over 64 entries (sorted in LDS by a bitmap over their entry
    range); with one row and 400 bags of up to 90 ids, a row of over 16384
    entries (the selection path); with 30000 bags of up to 20 ids over 30 or
    500 rows, buckets of 1025..16384 and of 65..1024 entries whose entries
    span more than the bitmap's 64 Ki (the bitonic sort); bit-identical on
    a second run."""
    _say(f"case: embed_bags_backward {dtype} dim={dim} M={M} T={T} rows={rows}")
    _, offsets, indices, _ = _bags(M * 17 + dim, M, T, rows, dim, n_dense, max_len)
    rng = np.random.Generator(np.random.PCG64(M + dim))
    x_ld = (n_dense + T * dim + 7) // 8 * 8
    dx = rng.normal(size=(M, x_ld)).astype(np.float32)
    if dtype == "bf16":
        dx = synth.round_to_bf16_values(dx)
    g, st = _run_bags_bwd(offsets, indices, dx, n_dense, rows, dim, dtype)
    assert st == 0
    ref = oracle.embed_bags_backward(offsets, indices, dx.astype(np.float64), n_dense, rows, dim)
    mag = oracle.embed_bags_backward(offsets, indices, np.abs(dx.astype(np.float64)), n_dense, rows, dim)
    # fp32 sums of the same bf16/fp32 inputs, within the rounding bound of a
    # sum of n terms in any order, (n - 1) 2^-24 times the sum of magnitudes
    # (at least 1e-6 of it), n the row's entry count
    n_r = np.zeros((T, rows), dtype=np.float64)
    for t in range(T):
        np.add.at(n_r[t], indices[offsets[t, 0]:offsets[t, -1]], 1.0)
    tol = np.maximum(1e-6, (n_r - 1.0) * 2.0 ** -24)[:, :, None]
    assert np.all(np.abs(g - ref) <= tol * mag + 1e-30)
    used = {(t, int(r)) for t in range(T) for r in indices[offsets[t, 0]:offsets[t, -1]]}
    for t in range(T):
        for r in range(rows):
            if (t, r) not in used:
                assert np.all(g[t, r] == 0.0)
    g2, _ = _run_bags_bwd(offsets, indices, dx, n_dense, rows, dim, dtype)
    assert np.array_equal(g.view(np.uint32), g2.view(np.uint32))


def test_embed_bags_backward_full_ctr_shape():
    """The CTR input stage's backward at full size (4096 rows, 26 tables of
    100000 x 64, Zipf(1.1) bags of 1..20 ids) with a bf16 dx: sampled rows
    against their sums written out from the data, total mass per table, and
    a bit-identical second run."""
    _say("case: embed_bags_backward full CTR shape")
    rng = np.random.Generator(np.random.PCG64(1))
    tabs = synth.CtrTables(rng)
    raw = synth.make_ctr_raw(tabs, 4096, rng)
    offsets, indices = raw["offsets"], raw["indices"]
    dx = synth.round_to_bf16_values(rng.normal(size=(4096, 1680)).astype(np.float32))
    g, st = _run_bags_bwd(offsets, indices, dx, 13, synth.CTR_ROWS, 64, "bf16")
    assert st == 0
    T = offsets.shape[0]
    bag_of = np.empty(int(offsets[-1, -1]), dtype=np.int64)
    for t in range(T):
        for m in range(4096):
            bag_of[offsets[t, m]:offsets[t, m + 1]] = m
    pick = np.random.Generator(np.random.PCG64(2))
    for _ in range(40):
        t = int(pick.integers(0, T))
        seg = indices[offsets[t, 0]:offsets[t, -1]]
        r = int(seg[pick.integers(0, seg.size)])            # a row some entry selects
        ent = np.nonzero(seg == r)[0] + offsets[t, 0]
        want = dx[bag_of[ent]][:, 13 + 64 * t: 13 + 64 * (t + 1)].astype(np.float64).sum(axis=0)
        mag = np.abs(dx[bag_of[ent]][:, 13 + 64 * t: 13 + 64 * (t + 1)].astype(np.float64)).sum(axis=0)
        assert np.all(np.abs(g[t, r] - want) <= 1e-6 * mag + 1e-30), (t, r)
    for t in range(T):
        lens = np.diff(offsets[t]).astype(np.float64)
        want = (lens[:, None] * dx[:, 13 + 64 * t: 13 + 64 * (t + 1)].astype(np.float64)).sum(axis=0)
        np.testing.assert_allclose(g[t].astype(np.float64).sum(axis=0), want, rtol=1e-4, atol=1e-2)
    g2, _ = _run_bags_bwd(offsets, indices, dx, 13, synth.CTR_ROWS, 64, "bf16")
    assert np.array_equal(g.view(np.uint32), g2.view(np.uint32))


def test_embed_bags_backward_invalid_entries_flagged():
    """Out-of-range ids and bag bounds are skipped and set the status word;
    the rows of every other entry are exact."""
    _say("case: embed_bags_backward invalid entries")
    _, offsets, indices, _ = _bags(43, 16, 3, 50, 64, 2, 5, allow_empty=False)
    rng = np.random.Generator(np.random.PCG64(44))
    dx = rng.normal(size=(16, 200)).astype(np.float32)
    bad_idx = indices.copy()
    bad_idx[offsets[1, 3]] = 50
    bad_idx[offsets[2, 7]] = -1
    g, st = _run_bags_bwd(offsets, bad_idx, dx, 2, 50, 64, "f32")
    assert st == 1
    keep = np.ones(indices.size, dtype=bool)
    keep[[offsets[1, 3], offsets[2, 7]]] = False
    # the oracle with the two invalid entries pointed at a scratch row past the table
    idx2 = np.where(keep, indices, 50)
    ref = oracle.embed_bags_backward(offsets, idx2, dx.astype(np.float64), 2, 51, 64)[:, :50]
    np.testing.assert_allclose(g, ref, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_lambda_block_is_frozen(dtype):
    """lambda_b = 0 (Eq. 2): the block's gradient is exactly zero, so Adam
    leaves its parameters bit-identical (m = v = 0, update 0/(0 + eps)); the
    other blocks still match the oracle."""
    _say(f"case: zero lambda, {dtype}")
    blocks = [{"input": "x", "layers": [("linear_relu", 40, 24), ("linear_relu", 24, 16)], "lam": 0.0},
              {"input": "x", "layers": [("linear_relu", 40, 32)], "lam": 1.0},
              {"input": "prev", "layers": [("linear_relu", 32, 8)], "lam": 0.0}]
    cfg = synth.custom(dtype, 97, 40, blocks, label_p=0.4)
    params, batches = synth.make_workload(cfg, 23, 3)
    _, g = run_gpu(cfg, params, batches, "overlap")
    init = [erase.pack_block(p) for p in params]
    for b in (0, 2):
        assert np.array_equal(g[-1]["params"][b].view(np.uint32), init[b].view(np.uint32)), b
        assert not np.any(g[-1]["m"][b]) and not np.any(g[-1]["v"][b]) and not np.any(g[-1]["grads"][b])
    if dtype == "f32":
        compare(cfg, g, run_oracle(cfg, params, batches), 1e-4)
    else:
        _say("  ", check_bf16(cfg, g, params, batches))


def test_maximum_block_and_layer_counts_fp32():
    """64 chained blocks (the most a context takes) and a 16-layer block."""
    _say("case: 64 chained blocks; a 16-layer block")
    blocks = [{"input": "x" if b == 0 else "prev", "layers": [("linear_relu", 6 if b == 0 else 5, 5)],
               "lam": 1.0} for b in range(64)]
    cfg = synth.custom("f32", 33, 6, blocks, label_p=0.5)
    params, batches = synth.make_workload(cfg, 29, 2)
    _, g = run_gpu(cfg, params, batches, "pipeline")
    _say("  ", check_f32(cfg, g, params, batches))
    widths = [9] + [7 if i % 2 else 11 for i in range(16)]
    blocks = [{"input": "x", "layers": [("linear_relu", widths[i], widths[i + 1]) for i in range(16)], "lam": 1.0}]
    cfg = synth.custom("f32", 45, 9, blocks, label_p=0.5)
    params, batches = synth.make_workload(cfg, 31, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    compare(cfg, g, run_oracle(cfg, params, batches), 1e-4)


def test_widest_hidden_layer_fp32():
    """A 65536-wide hidden layer (the widest a layer may be): its GEMMs have
    65536 output columns and a 65536-long contraction."""
    _say("case: 16 -> 65536 -> 48 fp32")
    blocks = [{"input": "x", "layers": [("linear_relu", 16, 65536), ("linear_relu", 65536, 48)], "lam": 1.0}]
    cfg = synth.custom("f32", 40, 16, blocks, label_p=0.5)
    params, batches = synth.make_workload(cfg, 37, 2)
    _, g = run_gpu(cfg, params, batches, "serial")
    compare(cfg, g, run_oracle(cfg, params, batches), 1e-4)


def test_long_ragged_batch_bf16():
    """70001 rows: ragged M tiles, and weight gradients whose split
    contraction ends in a ragged k-step."""
    _say("case: batch 70001 bf16")
    blocks = [{"input": "x", "layers": [("linear_relu", 24, 40), ("linear_relu", 40, 16)], "lam": 1.0},
              {"input": "prev", "layers": [("linear_relu", 16, 24)], "lam": 0.5}]
    cfg = synth.custom("bf16", 70001, 24, blocks, label_p=0.1)
    params, batches = synth.make_workload(cfg, 41, 2)
    _, g = run_gpu(cfg, params, batches, "pipeline")
    _say("  ", check_bf16(cfg, g, params, batches))


def test_deep_chain_multi_stream_matches_serial():
    """A chain with 4 backward streams: bit-identical to the serial schedule."""
    _say("case: deep_chain, 4 backward streams vs serial")
    cfg = synth.config("deep_chain", batch=512)
    params, batches = synth.make_workload(cfg, 7, 2)
    a = run_gpu(cfg, params, batches, "serial")[1]
    b = run_gpu(cfg, params, batches, "overlap", bwd_streams=4)[1]
    c = run_gpu(cfg, params, batches, "overlap_graph", bwd_streams=4)[1]
    assert_bit_identical(a, b)
    assert_bit_identical(a, c)


def test_ctr_mlp_full_size_vs_oracle():
    """The benchmarked workload itself (6 blocks, batch 4096, bf16), 2 steps,
    in the benchmark's headline schedule: PIPELINE with the backward work
    enqueued by the library's worker thread on 2 backward streams."""
    _say("case: ctr_mlp full size, pipeline+worker, 2 backward streams")
    cfg = synth.config("ctr_mlp")
    params, batches = synth.make_workload(cfg, 0, 2)
    tr = erase.Trainer(cfg, params, keep_grads=True, bwd_streams=2)
    tr.set_dispatch("worker")
    _, g = run_gpu(cfg, params, batches, "pipeline", trainer=tr)
    tr.close()
    _say("  ", check_bf16(cfg, g, params, batches))


def test_ctr_mlp_full_size_headline_schedule_bit_identical():
    """At the benchmarked size (6 blocks, batch 4096, bf16, 2 backward
    streams, worker dispatch), 6 PIPELINE steps enqueued back to back -- so
    the zero-padded input copies and the events of one step are reused while
    the previous step's backward may still run -- and a mix with
    OVERLAP_GRAPH and OVERLAP give the same bits as 6 SERIAL steps: losses of
    every step, and the final gradients, parameters and moments."""
    _say("case: ctr_mlp full size, pipeline+worker back to back vs serial")
    cfg = synth.config("ctr_mlp")
    params, batches = synth.make_workload(cfg, 19, 6)
    ref_l, ref = run_gpu_nosync(cfg, params, batches, ["serial"])
    for scheds in (["pipeline"], ["pipeline", "overlap_graph", "pipeline", "pipeline", "overlap", "pipeline"]):
        got_l, got = run_gpu_nosync(cfg, params, batches, scheds, bwd_streams=2, dispatch="worker")
        assert np.array_equal(ref_l.view(np.uint32), got_l.view(np.uint32)), scheds
        assert_bit_identical([ref], [got])


def test_x_in_place_matches_the_padded_copy():
    """The GEMMs reading the caller's zero-padded x in place give the same
    bits as the step that copies x into its workspace, in the serial and
    the headline schedule (pipeline, worker dispatch, 2 backward streams),
    over 3 back-to-back steps; cross layers read x0 in place too."""
    _say("case: x read in place vs padded copy")
    cfg = _ctr_small(batch=512, blocks=3)
    dcn = synth.config("ctr_dcn", batch=256, ctr_rows=5000)
    dcn["blocks"] = dcn["blocks"][:1]
    for c in (cfg, dcn):
        params, batches = synth.make_workload(c, 27, 3)
        ref_l, ref = run_gpu_nosync(c, params, batches, ["serial"])
        for scheds, disp in ((["serial"], "caller"), (["pipeline"], "worker")):
            import torch
            tr = erase.Trainer(c, params, keep_grads=True, bwd_streams=2, x_in_place=True)
            assert tr.ncfg.x_ld % 128 == 0
            tr.set_dispatch(disp)
            dev = [tr.device_batch(x, y) for (x, y) in batches]
            outs = [torch.zeros(len(c["blocks"]), dtype=torch.float32, device="cuda") for _ in batches]
            for i, (xd, yd) in enumerate(dev):
                tr.step(xd, yd, scheds[0], losses=outs[i], wait_current=(i == 0))
            tr.sync()
            p, m, v, g = tr.flat_state()
            tr.close()
            got_l = np.stack([o.cpu().numpy() for o in outs])
            assert np.array_equal(ref_l.view(np.uint32), got_l.view(np.uint32)), scheds
            assert_bit_identical([ref], [{"losses": got_l[-1], "params": p, "m": m, "v": v, "grads": g}])


def test_deep_chain_full_size_vs_oracle():
    _say("case: deep_chain full size")
    cfg = synth.config("deep_chain")
    params, batches = synth.make_workload(cfg, 0, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    _say("  ", check_bf16(cfg, g, params, batches))


def test_dcn_bf16_small_vs_oracle():
    _say("case: dcn bf16 small")
    blocks = [{"input": "x", "layers": [("cross", 200, 200), ("cross", 200, 200), ("linear_relu", 200, 128),
                                        ("linear_relu", 128, 64)], "lam": 1.0} for _ in range(2)]
    cfg = synth.custom("bf16", 300, 200, blocks, label_p=0.1)
    params, batches = synth.make_workload(cfg, 5, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    _say("  ", check_bf16(cfg, g, params, batches))


def test_ctr_dcn_bf16_small_vs_oracle():
    """The DCN workload's real shape (1677-wide cross layers on the CTR input,
    1677->1024->1024->512), ragged batch 300, 2 blocks."""
    _say("case: ctr_dcn bf16 batch=300")
    cfg = synth.config("ctr_dcn", batch=300, ctr_rows=5000)
    cfg["blocks"] = cfg["blocks"][:2]
    params, batches = synth.make_workload(cfg, 1, 2)
    _, g = run_gpu(cfg, params, batches, "overlap")
    _say("  ", check_bf16(cfg, g, params, batches))


def test_ctr_dcn_full_size_vs_oracle():
    """The DCN workload at full size (6 blocks, batch 16384, 1677-wide cross
    layers) in the overlapped schedule; blocks 0 and 5 are checked against the
    oracle (blocks read the shared input and are independent, so the oracle
    runs on just those two)."""
    _say("case: ctr_dcn full size, blocks 0 and 5 checked")
    cfg = synth.config("ctr_dcn")
    params, batches = synth.make_workload(cfg, 0, 1)
    _, g = run_gpu(cfg, params, batches, "overlap")
    sel = [0, 5]
    sub = dict(cfg)
    sub["blocks"] = [cfg["blocks"][i] for i in sel]
    gsub = [{k: (v[sel] if k == "losses" else [v[i] for i in sel]) for k, v in rec.items()} for rec in g]
    _say("  ", check_bf16(sub, gsub, [params[i] for i in sel], batches))


def test_nonfinite_input_is_reported():
    _say("case: non-finite input")
    cfg = synth.config("tiny")
    params, batches = synth.make_workload(cfg, 0, 1)
    x, y = batches[0]
    x = x.copy()
    x[3, 5] = np.nan
    tr = erase.Trainer(cfg, params)
    xd, yd = tr.device_batch(x, y)
    tr.step(xd, yd, "overlap")
    with pytest.raises(erase.EraseError) as ei:
        tr.sync()
    assert ei.value.status == erase.ERR_NONFINITE
    with pytest.raises(erase.EraseError) as ei:  # sticky
        tr.step(xd, yd, "overlap")
    assert ei.value.status == erase.ERR_STATE


def test_checkpoint_resume_bit_identical():
    _say("case: checkpoint/resume")
    cfg = _mixed_fp32(96)
    params, batches = synth.make_workload(cfg, 6, 4)
    _, full = run_gpu(cfg, params, batches, "overlap")
    tr, first = run_gpu(cfg, params, batches[:2], "overlap")
    p, m, v, _g = tr.state()
    t = tr.get_step()
    assert t == 2
    tr.close()
    tr2 = erase.Trainer(cfg, p, m=m, v=v, step=t)
    _, rest = run_gpu(cfg, p, batches[2:], "overlap", trainer=tr2)
    assert_bit_identical(full, first + rest)


def test_repeatable_across_contexts():
    _say("case: repeatability")
    cfg = _ctr_small(batch=512, blocks=2)
    params, batches = synth.make_workload(cfg, 9, 2)
    a = run_gpu(cfg, params, batches, "overlap_graph")[1]
    b = run_gpu(cfg, params, batches, "overlap_graph")[1]
    assert_bit_identical(a, b)


def test_kernel_timing_records():
    _say("case: kernel timing")
    cfg = _ctr_small(batch=512, blocks=2)
    params, batches = synth.make_workload(cfg, 9, 1)
    tr = erase.Trainer(cfg, params)
    xd, yd = tr.device_batch(*batches[0])
    tr.set_timing(True)
    tr.step(xd, yd, "overlap")
    tr.sync()
    recs = tr.read_timing()
    assert recs[0]["kind"] == "empty" and recs[0]["end_ms"] >= recs[0]["start_ms"]
    recs = recs[1:]
    # prologue + per block: 3 forward GEMMs (the last with the head and loss
    # in its epilogue: the last layer is 128 wide), 2 grouped backward GEMMs,
    # the first layer's weight gradient with every Adam update of the block
    assert len(recs) == 1 + 2 * 6, [r["kind"] for r in recs]
    assert [r["kind"] for r in recs].count("wgrad_adam_kg2") == 2
    # (a forward GEMM of at most one workgroup per CU runs with two k-groups)
    assert [r["kind"].replace("_kg2", "") for r in recs[1:4]] == ["fwd_gemm", "fwd_gemm", "fwd_head_gemm"]
    assert all(r["end_ms"] >= r["start_ms"] >= 0 for r in recs)
    assert {r["stream"] for r in recs if r["kind"] in ("wgrad_gemm", "wgrad_gemm_kg2", "wgrad_adam_kg2", "bwd_gemm",
                                                        "adam")} == {1}
    tr2 = erase.Trainer(cfg, params, bwd_streams=2)
    tr2.set_timing(True)
    tr2.step(*tr2.device_batch(*batches[0]), "overlap")
    tr2.sync()
    r2 = tr2.read_timing()[1:]
    assert {r["stream"] for r in r2 if r["kind"] == "wgrad_adam_kg2"} == {1, 2}
    assert {r["stream"] for r in recs if r["kind"] in ("fwd_gemm", "fwd_gemm_kg2", "prologue")} == {0}
    # the last layer with its fused head runs on the backward stream in the
    # ERASE order (no later block reads the block's output), on the forward
    # stream in the serial one
    assert {r["stream"] for r in recs if r["kind"] == "fwd_head_gemm"} == {1}
    tr.step(xd, yd, "serial")
    tr.sync()
    assert {r["stream"] for r in tr.read_timing()[1:] if r["kind"] == "fwd_head_gemm"} == {0}
    with pytest.raises(erase.EraseError):
        tr.step(xd, yd, "overlap_graph")
    # a standalone head (256-wide chain blocks) runs on the backward stream in
    # the ERASE order, on the forward stream in the serial one
    cc = synth.config("deep_chain", batch=256)
    cc["blocks"] = cc["blocks"][:3]
    pc, bc = synth.make_workload(cc, 9, 1)
    tc = erase.Trainer(cc, pc)
    xc, yc = tc.device_batch(*bc[0])
    tc.set_timing(True)
    for sched, want in (("overlap", {1}), ("serial", {0})):
        tc.step(xc, yc, sched)
        tc.sync()
        rc = tc.read_timing()[1:]
        assert {r["stream"] for r in rc if r["kind"] == "head_bce"} == want, sched
        assert len([r for r in rc if r["kind"] == "head_bce"]) == 3
    tc.close()
