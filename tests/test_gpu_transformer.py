"""GPU parity of the detached small-transformer step (include/erase_tf.h)
against the CPU oracle (oracle/transformer_oracle.py), through the C ABI.

bf16 bounds (tests/gpu_util.bf16_gate), norm-wise per tensor and plain
relative per loss: 2e-2 against the oracle that rounds to bf16 the tensors
the GPU stores in bf16 (on later steps max(2e-2, 1.5 e_acc), e_acc = that
oracle's own float32-vs-float64 spread); against the float64 oracle
max(2e-2, 1.5 e_bf), e_bf = the emulating oracle's distance from float64."""
import math

import numpy as np
import pytest

from oracle import transformer_oracle as to
from paper_2608_18469_amd import synth_tf
from tests.gpu_util import bf16_gate

pytestmark = pytest.mark.gpu

FIELDS = ("losses", "grads", "params", "m", "v")


def _trainer(cfg, params, **kw):
    from paper_2608_18469_amd import erase_tf
    return erase_tf.TfTrainer(cfg, params, **kw)


def _gpu_run(cfg, params, batches, schedule="serial", tr=None):
    tr = tr or _trainer(cfg, params)
    recs = []
    for tok in batches:
        t = tr.device_tokens(tok)
        tr.step(t, schedule)
        tr.sync()
        p, m, v, g = tr.flat_state()
        recs.append({"losses": tr.losses.cpu().numpy().copy(), "params": p, "m": m, "v": v, "grads": g})
    return tr, recs


def _oracle_run(cfg, params, batches, emulate_bf16=False, dtype=np.float64):
    m = synth_tf.zero_state(params)
    v = synth_tf.zero_state(params)
    p, t, recs = params, 0, []
    for tok in batches:
        r = to.tf_step(cfg, p, m, v, t, tok, emulate_bf16=emulate_bf16, dtype=dtype)
        p, m, v, t = r["params"], r["m"], r["v"], r["t"]
        print(f"[tf oracle] step {t} done (emulate_bf16={emulate_bf16}, {np.dtype(dtype).name})", flush=True)
        pk = lambda tree: [synth_tf.pack_block(cfg, b, tree[b]) for b in range(cfg["layers"])]
        recs.append({"losses": np.array(r["losses"]), "params": pk(p), "m": pk(m), "v": pk(v), "grads": pk(r["grads"])})
    return recs


def _rel(a, b):
    a, b = np.asarray(a, np.float64).reshape(-1), np.asarray(b, np.float64).reshape(-1)
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / nb if nb > 0 else np.linalg.norm(a - b)


def _worst(cfg, got, ref):
    out = {}
    for k in FIELDS:
        w = 0.0
        for g, r in zip(got, ref):
            if k == "losses":
                w = max(w, float(np.max(np.abs(g[k] - r[k]) / np.abs(r[k]))))
                continue
            for b in range(cfg["layers"]):
                G = synth_tf.unpack_block(cfg, b, np.asarray(g[k][b]))
                R = synth_tf.unpack_block(cfg, b, np.asarray(r[k][b], np.float64))
                for name in G:
                    w = max(w, _rel(G[name], R[name]))
        out[k] = w
    return out


def _check_bf16(cfg, gpu, params, batches, tol=2e-2, slack=1.5):
    """bf16 parity against the float64 and the bf16-emulating oracles
    (tests/gpu_util.bf16_gate: flat tol against the emulating oracle on the
    first step)."""
    r64 = _oracle_run(cfg, params, batches)
    rbf = _oracle_run(cfg, params, batches, emulate_bf16=True)
    rbf32 = _oracle_run(cfg, params, batches, emulate_bf16=True, dtype=np.float32) if len(batches) > 1 else None
    return bf16_gate(lambda a, b: _worst(cfg, a, b), gpu, r64, rbf, rbf32, tol, slack, "tf")


def _bits_equal(a, b):
    for ra, rb in zip(a, b):
        assert np.array_equal(ra["losses"].view(np.uint32), rb["losses"].view(np.uint32))
        for k in ("params", "m", "v", "grads"):
            for x, y in zip(ra[k], rb[k]):
                assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), k


def test_tf_small_two_steps_match_oracle():
    cfg = synth_tf.tf_config("tf_small")
    params, batches = synth_tf.make_workload(cfg, seed=0, n_batches=2)
    print("[tf] tf_small serial, 2 steps", flush=True)
    _, gpu = _gpu_run(cfg, params, batches, "serial")
    _check_bf16(cfg, gpu, params, batches)


def test_tf_overlap_is_bit_identical_to_serial():
    cfg = synth_tf.tf_config("tf_small", layers=3)
    params, batches = synth_tf.make_workload(cfg, seed=1, n_batches=2)
    print("[tf] tf_small serial vs overlap", flush=True)
    _, a = _gpu_run(cfg, params, batches, "serial")
    _, b = _gpu_run(cfg, params, batches, "overlap")
    _bits_equal(a, b)


def test_tf_ragged_shapes_match_oracle():
    # T not a multiple of the 64-row attention block, B*T not a multiple of
    # the 128-row GEMM tile, V a multiple of 64 only, one head
    cfg = synth_tf.tf_config("tf_tiny", vocab=192, d=64, heads=1, layers=2, seq=100, batch=3)
    params, batches = synth_tf.make_workload(cfg, seed=2, n_batches=1)
    print("[tf] ragged T=100 B=3 V=192 d=64", flush=True)
    _, gpu = _gpu_run(cfg, params, batches, "overlap")
    _check_bf16(cfg, gpu, params, batches)


def test_tf_single_position_and_four_heads():
    cfg = synth_tf.tf_config("tf_tiny", vocab=256, d=256, heads=4, layers=2, seq=1, batch=5)
    params, batches = synth_tf.make_workload(cfg, seed=3, n_batches=1)
    print("[tf] T=1 B=5 d=256 H=4", flush=True)
    _, gpu = _gpu_run(cfg, params, batches, "serial")
    _check_bf16(cfg, gpu, params, batches)


def test_tf_forward_intermediates_match_oracle():
    """Block 1's stored activations against the bf16-emulating oracle's."""
    cfg = synth_tf.tf_config("tf_small")
    params, batches = synth_tf.make_workload(cfg, seed=4, n_batches=1)
    tr, _ = _gpu_run(cfg, params, batches, "serial")
    caches, _, _ = to._forward(cfg, params, batches[0], True, np.float64)
    c = caches[0]
    N, d = cfg["batch"] * cfg["seq"], cfg["d"]
    for name, ref, cols in (("qkv", None, 3 * d), ("o", c["o"], d), ("a1", c["a1"], d), ("u", c["u"], 4 * d),
                            ("g", c["g"], 4 * d), ("z", c["z"], d), ("hn", c["hn"], d)):
        got = tr.tensor(0, name, N, cols)
        if ref is None:
            from oracle.transformer_oracle import _unheads
            ref = np.concatenate([_unheads(c["q"]), _unheads(c["k"]), _unheads(c["v"])], axis=1)
        e = _rel(got, ref)
        print(f"[tf] block 0 {name}: rel {e:.2e}", flush=True)
        assert e < 2e-2, (name, e)
    lse = tr.tensor(0, "lse", cfg["batch"] * cfg["heads"], cfg["seq"], dtype="f32")
    assert np.all(np.isfinite(lse))


def test_tf_zero_head_closed_form():
    cfg = synth_tf.tf_config("tf_small")
    params, batches = synth_tf.make_workload(cfg, seed=5, n_batches=1)
    for p in params:
        p["wh"] = np.zeros_like(p["wh"])
    _, gpu = _gpu_run(cfg, params, batches, "overlap")
    lv = math.log(cfg["vocab"])
    assert np.all(np.abs(gpu[0]["losses"] - lv) <= 1e-6 * lv), gpu[0]["losses"]
    for b in range(cfg["layers"]):
        G = synth_tf.unpack_block(cfg, b, gpu[0]["grads"][b])
        for k in ("wqkv", "wo", "w1", "w2") + (("emb",) if b == 0 else ()):
            assert np.all(G[k] == 0.0), (b, k)


def test_tf_invalid_token_is_reported():
    from paper_2608_18469_amd import erase
    cfg = synth_tf.tf_config("tf_small", layers=1)
    params, batches = synth_tf.make_workload(cfg, seed=6, n_batches=1)
    tok = batches[0].copy()
    tok[1, 5] = cfg["vocab"]
    tr = _trainer(cfg, params)
    tr.step(tr.device_tokens(tok), "serial")
    with pytest.raises(erase.EraseError) as ei:
        tr.sync()
    assert ei.value.status == erase.ERR_INVALID_ARG
    tr.close()


def _bf16_view(tr, block, name, rows):
    """Device view [rows][pitch] (bf16) of a stored tensor, without a copy."""
    import ctypes
    from paper_2608_18469_amd import erase_tf
    torch = tr.torch
    p, ld = ctypes.c_void_p(), ctypes.c_int64(0)
    assert erase_tf.lib().erase_tf_tensor(tr.ctx, block, erase_tf.TENSORS[name], ctypes.byref(p),
                                          ctypes.byref(ld)) == 0
    tr.sync()
    off = p.value - tr.ws.data_ptr()
    assert 0 <= off and off + rows * ld.value * 2 <= tr.ws.numel()
    return tr.ws[off:off + rows * ld.value * 2].view(torch.bfloat16).view(rows, ld.value)


def test_tf_c5_full_size_sampled():
    """The full small-transformer shape (V 32768, d 512, 8 heads, 8 layers,
    T 1024, B 16) in the launch configuration the benchmark times: serial and
    overlapped steps agree bit for bit; block 1's stored output and attention
    statistics of the first sequence match the oracle run on that sequence
    alone; losses are near log V at initialisation."""
    cfg = synth_tf.tf_config("tf_c5")
    params, batches = synth_tf.make_workload(cfg, seed=0, n_batches=1)
    print("[tf] c5 serial", flush=True)
    tra, a = _gpu_run(cfg, params, batches, "serial")
    T, d = cfg["seq"], cfg["d"]
    z0 = tra.tensor(0, "z", T, d)
    o0 = tra.tensor(0, "o", T, d)
    lse0 = tra.tensor(0, "lse", cfg["heads"], T, dtype="f32")
    V = cfg["vocab"]
    # after the step: the head's exponentials with the target entry minus the
    # row sum, and the row scale; their product is the logit gradient
    dl0 = _bf16_view(tra, 0, "logits", T)[:, :V].float().cpu().numpy()
    dl0 = dl0 * tra.tensor(0, "rowscale", 1, T, dtype="f32")[0][:, None]
    tra.close()
    del tra
    print("[tf] c5 overlap", flush=True)
    trb, b = _gpu_run(cfg, params, batches, "overlap")
    trb.close()
    _bits_equal(a, b)
    losses = a[0]["losses"]
    lv = math.log(cfg["vocab"])
    assert np.all(np.abs(losses - lv) < 1.0), losses
    one = dict(cfg, batch=1)
    caches, _, _ = to._forward(one, [{k: params[0][k] for k in params[0]}], batches[0][:1], True, np.float64)
    c = caches[0]
    ez, eo = _rel(z0, c["z"]), _rel(o0, c["o"])
    print(f"[tf] c5 sequence 0: z rel {ez:.2e}, o rel {eo:.2e}", flush=True)
    assert ez < 2e-2 and eo < 2e-2
    # lse of head h, row t: log sum_j exp(s_tj) over j <= t, from the oracle's q, k
    q, k = c["q"][0], c["k"][0]
    s = np.matmul(q, np.swapaxes(k, -1, -2)) / 8.0
    s = np.where(np.triu(np.ones((T, T), bool), 1), -np.inf, s)
    mx = s.max(-1, keepdims=True)
    ref = (mx + np.log(np.exp(s - mx).sum(-1, keepdims=True)))[..., 0]
    assert np.max(np.abs(lse0 - ref)) < 5e-2, np.max(np.abs(lse0 - ref))
    # the head of block 1 on sequence 0: logits GEMM, row sums and
    # normaliser, through the logit gradient lam (softmax - onehot) / N
    x = c["logits"]
    p = np.exp(x - x.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    p[np.arange(T), np.asarray(batches[0][0, 1:T + 1])] -= 1.0
    p *= float(cfg.get("lam", 1.0)) / (cfg["batch"] * T)
    e = _rel(dl0, p)
    print(f"[tf] c5 sequence 0 logit gradient: rel {e:.2e}", flush=True)
    assert e < 2e-2, e


def _plan(cfg, params, tok):
    """(kind, GEMM, tile rows, tile columns, split) of every GEMM launch of
    one serial step: the launch configuration the shape selects."""
    tr = _trainer(cfg, params, keep_grads=False)
    tr.set_timing(True)
    tr.step(tr.device_tokens(tok), "serial")
    tr.sync()
    plan = {(r["kind"], r["layer"], r["tile_m"], r["tile_n"], r["split"]) for r in tr.read_timing()[1:]
            if r["kind"].endswith("gemm")}
    tr.close()
    return plan


@pytest.mark.timeout(900)
def test_tf_c5_kernel_classes_full_step_vs_oracle():
    """One whole step at a shape with the full model's launch configuration
    (16 sequences of 1024 tokens, width 512, 8 heads, vocabulary 16384, 2
    layers): every GEMM launch takes the tile, k-group and split of the
    benchmarked 8-layer, 32768-word model (among them the two k-group
    128x128 grouped vocabulary backward, the 256x256 logits kernel, the
    64x128 MLP-up and MLP-down input-gradient kernels, and the 128x128
    forward tiles) -- and
    losses, gradients, parameters and both Adam moments of both blocks (the
    second reads the first's output) match the oracles."""
    c5 = synth_tf.tf_config("tf_c5")
    cfg = synth_tf.tf_config("tf_c5", vocab=16384, layers=2)
    params, batches = synth_tf.make_workload(cfg, seed=0, n_batches=1)
    p5, b5 = synth_tf.make_workload(c5, seed=0, n_batches=1)
    print("[tf] launch plans of the full model and of V 16384, 2 layers", flush=True)
    want, got = _plan(c5, p5, b5[0]), _plan(cfg, params, batches[0])
    del p5, b5
    print(f"[tf] launch plan: {sorted(got)}", flush=True)
    assert got == want, (sorted(got ^ want))
    # the vocabulary head: 256x256 logits tiles, one grouped two k-group
    # 128x128 launch for both of its gradients
    assert ("bwd_gemm", 4, 128, 128, 1) in got and ("fwd_gemm", 4, 256, 256, 1) in got
    print("[tf] V 16384, 2 layers: GPU step", flush=True)
    tr, gpu = _gpu_run(cfg, params, batches, "serial")
    tr.close()
    print("[tf] V 16384, 2 layers: oracles (about a minute each)", flush=True)
    _check_bf16(cfg, gpu, params, batches)


def test_tf_logits_tiles_uneven_over_the_persistent_grid():
    """The 256x256 logits kernel runs one persistent workgroup per CU over
    its tiles: here 9 x 37 = 333 tiles for 256 workgroups, so some walk two
    tiles and the rest one (the next tile's first k-step and reference
    logits are loaded during the current tile's last k-step).  The step
    matches the oracles, and OVERLAP gives the same bits as SERIAL."""
    cfg = synth_tf.tf_config("tf_tiny", vocab=37 * 256, d=128, heads=2, layers=1, seq=1152, batch=2)
    params, batches = synth_tf.make_workload(cfg, seed=12, n_batches=1)
    plan = _plan(cfg, params, batches[0])
    print(f"[tf] N 2304, V 9472, d 128: launch plan {sorted(plan)}", flush=True)
    assert ("fwd_gemm", 4, 256, 256, 1) in plan
    _, a = _gpu_run(cfg, params, batches, "serial")
    _, b = _gpu_run(cfg, params, batches, "overlap")
    _bits_equal(a, b)
    _check_bf16(cfg, a, params, batches)


@pytest.mark.timeout(900)
def test_tf_c5_full_size_block1_vs_oracle():
    """The full model (V 32768, d 512, 8 heads, 8 layers, 16 x 1024 tokens)
    in the launch configuration the benchmark times: block 1 -- embedding,
    attention, MLP, its RMSNorm + 32768-word head, every gradient, the Adam
    update and the loss -- against the oracles run on that block alone (later
    blocks send it nothing: the cut of Eq. 1)."""
    cfg = synth_tf.tf_config("tf_c5")
    params, batches = synth_tf.make_workload(cfg, seed=0, n_batches=1)
    print("[tf] c5 full size: GPU step", flush=True)
    tr, rec = _gpu_run(cfg, params, batches, "serial")
    tr.close()
    one = dict(cfg, layers=1)
    sub = [{"losses": r["losses"][:1], **{k: r[k][:1] for k in ("params", "m", "v", "grads")}} for r in rec]
    print("[tf] c5 full size: block 1 oracles (one to two minutes each)", flush=True)
    _check_bf16(one, sub, params[:1], batches)


def test_tf_checkpoint_resume_is_bit_identical():
    """Two steps in one run equal one step, a save of params / m / v / t, a
    fresh context resumed from them, and a second step; also after the
    caller rewrites the parameters and refreshes the weight copies."""
    from paper_2608_18469_amd import erase_tf
    cfg = synth_tf.tf_config("tf_small")
    params, batches = synth_tf.make_workload(cfg, seed=7, n_batches=2)
    _, full = _gpu_run(cfg, params, batches, "overlap")
    tr1, one = _gpu_run(cfg, params, batches[:1], "overlap")
    assert tr1.get_step() == 1
    unpack = lambda flat: [synth_tf.unpack_block(cfg, b, flat[b]) for b in range(cfg["layers"])]
    p1, m1, v1 = unpack(one[0]["params"]), unpack(one[0]["m"]), unpack(one[0]["v"])
    tr1.close()
    tr2 = erase_tf.TfTrainer(cfg, p1, m=m1, v=v1, step=1)
    _, resumed = _gpu_run(cfg, p1, batches[1:], "overlap", tr=tr2)
    _bits_equal(full[1:], resumed)
    # overwrite the parameters in place, refresh the copies, step again
    for b in range(cfg["layers"]):
        tr2.param[b].copy_(tr2.torch.from_numpy(synth_tf.pack_block(cfg, b, p1[b])).to(tr2.dev))
        tr2.m[b].copy_(tr2.torch.from_numpy(synth_tf.pack_block(cfg, b, m1[b])).to(tr2.dev))
        tr2.v[b].copy_(tr2.torch.from_numpy(synth_tf.pack_block(cfg, b, v1[b])).to(tr2.dev))
    tr2.torch.cuda.synchronize()
    tr2.set_step(1)
    tr2.refresh_weights()
    _, again = _gpu_run(cfg, p1, batches[1:], "overlap", tr=tr2)
    _bits_equal(full[1:], again)
    tr2.close()


def test_tf_timing_records():
    cfg = synth_tf.tf_config("tf_small", layers=2)
    params, batches = synth_tf.make_workload(cfg, seed=8, n_batches=1)
    tr = _trainer(cfg, params)
    t = tr.device_tokens(batches[0])
    tr.set_timing(True)
    for sched in ("serial", "overlap"):
        tr.step(t, sched)
        tr.sync()
        recs = tr.read_timing()
        assert recs[0]["kind"] == "empty"
        kinds = {r["kind"] for r in recs[1:]}
        assert {"prologue", "embed", "rms_fwd", "fwd_gemm", "attn_fwd", "head_norm", "rms_bwd", "attn_bwd",
                "adam", "emb_grad"} <= kinds, kinds
        assert any(k in kinds for k in ("bwd_gemm", "wgrad_gemm"))
        for r in recs[1:]:
            assert r["end_ms"] >= r["start_ms"] >= 0.0
        streams = {r["stream"] for r in recs[1:]}
        assert streams == ({0} if sched == "serial" else {0, 1}), streams
        # per block: the forward body on stream 0, the head on the backward stream when overlapped
        # the normaliser and the recomputation of out-of-range rows: two launches per block
        heads = [r for r in recs[1:] if r["kind"] == "head_norm"]
        assert len(heads) == 2 * cfg["layers"] and all(r["stream"] == (0 if sched == "serial" else 1) for r in heads)
        assert sorted(r["layer"] for r in heads) == [0] * cfg["layers"] + [1] * cfg["layers"]
    tr.set_timing(False)
    tr.close()


def test_tf_head_rows_out_of_range():
    """Rows whose exponentials relative to the target logit sum past 2^60
    (row loss above 60 ln 2) take the recomputation with the row's exact
    maximum; the others the fast path.  A head weight 32 times its initial
    scale gives logits spread over about +-60, so both kinds of rows occur
    (checked on the oracle's row losses).  Compared with the float64 oracle:
    the bf16 emulation's exponentials relative to the target logit overflow
    bf16 on such rows, so it does not model them."""
    cfg = synth_tf.tf_config("tf_small", layers=1, seq=64)
    params, batches = synth_tf.make_workload(cfg, seed=12, n_batches=1)
    params[0]["wh"] = np.asarray(params[0]["wh"]) * 32.0  # a power of two: still bf16 values
    tok = batches[0]
    caches, _, tgt = to._forward(cfg, params, tok, False, np.float64)
    rows, _ = to.softmax_xent(caches[0]["logits"], tgt)
    far = int(np.sum(rows > 42.0))
    near = int(np.sum(rows < 40.0))
    print(f"[tf] head out-of-range rows: {far} above, {near} below of {rows.size}", flush=True)
    assert far > 0 and near > 0
    _, gpu = _gpu_run(cfg, params, batches, "serial")
    r64 = _oracle_run(cfg, params, batches)
    w = _worst(cfg, gpu, r64)
    print(f"[tf] head out-of-range rows vs float64: {w}", flush=True)
    assert all(w[k] < 2e-2 for k in FIELDS), w


def test_tf_widest_model():
    """The widest model the ABI accepts: d 4096 = 64 heads of 64 (RMSNorm and
    embedding-gradient rows at their maximum width)."""
    cfg = synth_tf.tf_config("tf_tiny", vocab=64, d=4096, heads=64, layers=1, seq=3, batch=2)
    params, batches = synth_tf.make_workload(cfg, seed=9, n_batches=1)
    print("[tf] d=4096 H=64", flush=True)
    _, gpu = _gpu_run(cfg, params, batches, "overlap")
    _check_bf16(cfg, gpu, params, batches)


def test_tf_long_sequence():
    cfg = synth_tf.tf_config("tf_tiny", vocab=128, d=64, heads=1, layers=2, seq=2048, batch=1)
    params, batches = synth_tf.make_workload(cfg, seed=10, n_batches=1)
    print("[tf] T=2048", flush=True)
    _, gpu = _gpu_run(cfg, params, batches, "overlap")
    _check_bf16(cfg, gpu, params, batches)


def test_tf_repeated_tokens_embedding_gradient():
    """One token at almost every position: its bucket (about 500 positions)
    takes the embedding gradient's ordering path for buckets over 64; the
    rest of the rows are empty or small."""
    cfg = synth_tf.tf_config("tf_tiny", vocab=128, d=128, heads=2, layers=1, seq=256, batch=2)
    params, batches = synth_tf.make_workload(cfg, seed=11, n_batches=1)
    tok = batches[0].copy()
    rng = np.random.Generator(np.random.PCG64(12))
    mask = rng.random(tok.shape) < 0.97
    tok[mask] = 7
    print("[tf] repeated token", flush=True)
    _, gpu = _gpu_run(cfg, params, [tok], "serial")
    _check_bf16(cfg, gpu, params, [tok])
    _, again = _gpu_run(cfg, params, [tok], "overlap")
    _bits_equal(gpu, again)
