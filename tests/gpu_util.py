"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
and the CPU oracle on the same seeded inputs, and compare per tensor."""
import sys

import numpy as np

import oracle
from paper_2608_18469_amd import erase, synth


def leaves(tree):
    out = []
    for (W, b) in tree["layers"]:
        out += [np.asarray(W), np.asarray(b)]
    out += [np.asarray(tree["head"][0]), np.asarray(tree["head"][1])]
    return out


def rel(a, b):
    a = np.asarray(a, dtype=np.float64).reshape(-1)
    b = np.asarray(b, dtype=np.float64).reshape(-1)
    nb = np.linalg.norm(b)
    d = np.linalg.norm(a - b)
    return d / nb if nb > 0 else d


def run_gpu(cfg, params, batches, schedule="overlap", keep_grads=True, trainer=None, bwd_streams=1):
    """Step the HIP path over `batches`; return per-step records."""
    tr = trainer or erase.Trainer(cfg, params, keep_grads=keep_grads, bwd_streams=bwd_streams)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    recs = []
    for (xd, yd) in dev:
        tr.step(xd, yd, schedule)
        tr.sync()
        p, m, v, g = tr.flat_state()
        recs.append({"losses": tr.losses.cpu().numpy().copy(), "params": p, "m": m, "v": v, "grads": g})
    return tr, recs


def run_gpu_nosync(cfg, params, batches, schedules, bwd_streams=1, dispatch="caller"):
    """Enqueue one step per batch (schedules[i % len] for step i) without
    synchronizing in between, then sync once; returns the per-step losses and
    the final state as one record list of length 1 plus the losses."""
    import torch
    tr = erase.Trainer(cfg, params, keep_grads=True, bwd_streams=bwd_streams)
    tr.set_dispatch(dispatch)
    dev = [tr.device_batch(x, y) for (x, y) in batches]
    outs = [torch.zeros(len(cfg["blocks"]), dtype=torch.float32, device="cuda") for _ in batches]
    for i, (xd, yd) in enumerate(dev):
        tr.step(xd, yd, schedules[i % len(schedules)], losses=outs[i], wait_current=(i == 0))
    tr.sync()
    p, m, v, g = tr.flat_state()
    losses = np.stack([o.cpu().numpy() for o in outs])
    tr.close()
    return losses, {"losses": losses[-1], "params": p, "m": m, "v": v, "grads": g}


def run_oracle(cfg, params, batches, emulate_bf16=False, t0=0, m=None, v=None, detach=True, dtype=np.float64):
    m = m or synth.zero_state(params)
    v = v or synth.zero_state(params)
    p, t = params, t0
    recs = []
    for (x, y) in batches:
        r = oracle.step(cfg, p, m, v, t, x, y, emulate_bf16=emulate_bf16, detach=detach, dtype=dtype)
        p, m, v, t = r["params"], r["m"], r["v"], r["t"]
        recs.append({"losses": np.array(r["losses"]),
                     "params": [erase.pack_block(q) for q in p],
                     "m": [erase.pack_block(q) for q in m],
                     "v": [erase.pack_block(q) for q in v],
                     "grads": [erase.pack_block(q) for q in r["grads"]],
                     "tree_params": p})
    return recs


FIELDS = ("losses", "grads", "params", "m", "v")


def worst_errors(cfg, gpu, ref, what=FIELDS):
    """Worst relative error per field over steps and block leaves (norm-wise
    per tensor, plain relative per loss)."""
    worst = {}
    for k in what:
        w = 0.0
        for g, r in zip(gpu, ref):
            if k == "losses":
                w = max(w, float(np.max(np.abs(g[k] - r[k]) / np.maximum(np.abs(r[k]), 1e-30))))
                continue
            for b, blk in enumerate(cfg["blocks"]):
                gt = erase.unpack_block(blk, np.asarray(g[k][b]))
                rt = erase.unpack_block(blk, np.asarray(r[k][b], dtype=np.float64))
                for A, B in zip(leaves(gt), leaves(rt)):
                    w = max(w, rel(A, B))
        worst[k] = w
    return worst


def compare(cfg, gpu, ref, tol, what=FIELDS):
    """Assert every field's worst relative error is within `tol`."""
    worst = worst_errors(cfg, gpu, ref, what)
    bad = {k: v for k, v in worst.items() if not v <= tol}
    assert not bad, f"tolerance {tol} exceeded: {worst}"
    return worst


def check_f32(cfg, gpu, params, batches, tol=1e-4, slack=2.0):
    """fp32 parity for deep compositions: the float64 oracle, within
    max(tol, slack * e) per field, where e is the float32 oracle's own
    distance from float64.  Through tens of chained blocks float32 rounding
    compounds (each block reads the previous block's rounded output), so a
    correct float32 step can sit above 1e-4 from float64; e measures that on
    the same inputs."""
    ref = run_oracle(cfg, params, batches)
    e = worst_errors(cfg, run_oracle(cfg, params, batches, dtype=np.float32), ref)
    got = worst_errors(cfg, gpu, ref)
    bad = {k: (got[k], max(tol, slack * e[k])) for k in got if not got[k] <= max(tol, slack * e[k])}
    assert not bad, f"fp32 bound exceeded (error, bound): {bad}; float32 oracle error {e}"
    return got, e


def bf16_gate(worst, gpu, r64, rbf, rbf32, tol=2e-2, slack=1.5, label="bf16"):
    """The bf16 parity gate, step by step, for any workload.

    ``worst(a, b)`` gives the worst relative error per field between two
    record lists.  Three oracle runs on the same inputs: ``r64`` in float64,
    ``rbf`` rounding to bf16 exactly the tensors the GPU stores in bf16, and
    ``rbf32`` the same rounding with float32 arithmetic (used from the second
    step on; None for a one-step run).

    * GPU vs the bf16-emulating oracle: flat ``tol`` on the first step, where
      both start from the same state.  A later step starts from the previous
      update, which on any float32 implementation differs from the float64
      one by rounding: Adam's first update is about lr * sign(g), so elements
      with tiny gradients move by up to 2 lr apart, move the bf16 copy of a
      weight by an ulp, and flip the ReLU masks of pre-activations that sit
      closer to zero than that.  How far that alone carries is measured, not
      assumed: ``e_acc``, the float32 emulating oracle's distance from the
      float64 one at that step.  Bound: max(tol, slack * e_acc).
    * GPU vs the float64 oracle: max(tol, slack * e_bf), where e_bf is the
      emulating oracle's own distance from float64 (what bf16 storage itself
      costs on this workload).
    Prints every step's errors and bounds; returns them.
    """
    rep = []
    bad = []
    for s in range(len(gpu)):
        e_acc = worst([rbf32[s]], [rbf[s]]) if s > 0 else None
        e_bf = worst([rbf[s]], [r64[s]])
        w_em = worst([gpu[s]], [rbf[s]])
        w_64 = worst([gpu[s]], [r64[s]])
        row = {}
        for k in w_em:
            b_em = tol if s == 0 else max(tol, slack * e_acc[k])
            b_64 = max(tol, slack * e_bf[k])
            row[k] = {"vs_emul": float(w_em[k]), "bound_emul": float(b_em), "vs_f64": float(w_64[k]),
                      "bound_f64": float(b_64), "emul_f32_vs_f64": None if e_acc is None else float(e_acc[k]),
                      "emul_vs_f64": float(e_bf[k])}
            if not (w_em[k] <= b_em and w_64[k] <= b_64):
                bad.append((s, k, row[k]))
        rep.append(row)
        print(f"[{label} parity] step {s + 1}: " + "; ".join(
            f"{k} emul {v['vs_emul']:.2e}/{v['bound_emul']:.2e} f64 {v['vs_f64']:.2e}/{v['bound_f64']:.2e}"
            for k, v in row.items()), file=sys.stderr, flush=True)
    assert not bad, f"{label} parity (step, field, errors and bounds): {bad}"
    return rep


def check_bf16(cfg, gpu, params, batches, tol=2e-2, slack=1.5, detach=True):
    """bf16 parity of a detached-block run against the oracle: ``bf16_gate``."""
    r64 = run_oracle(cfg, params, batches, detach=detach)
    rbf = run_oracle(cfg, params, batches, emulate_bf16=True, detach=detach)
    rbf32 = (run_oracle(cfg, params, batches, emulate_bf16=True, detach=detach, dtype=np.float32)
             if len(batches) > 1 else None)
    return bf16_gate(lambda a, b: worst_errors(cfg, a, b), gpu, r64, rbf, rbf32, tol, slack, cfg.get("name", "bf16"))


def assert_bit_identical(a, b):
    for ra, rb in zip(a, b):
        assert np.array_equal(ra["losses"].view(np.uint32), rb["losses"].view(np.uint32))
        for k in ("params", "m", "v", "grads"):
            for x, y in zip(ra[k], rb[k]):
                if x is None:
                    assert y is None
                    continue
                assert np.array_equal(x.view(np.uint32), y.view(np.uint32)), k
