"""Fused-node priorities and the ready-queue order on the device
(hs_priority after hs_dedup) against the oracle, bit for bit: phi* and pi
(fp64 bits) and the order, on the 1M-row workload's window, on the
chunk-dedup workload's 262,144 requests (56k fused nodes: several sorted
chunks and merge passes), with host and device distinct counts, all-equal
priorities (order = group order), and a single fused node."""
import numpy as np
import pytest
import torch

import oracle
from oracle import priority as pr
import synth
from gpu_harness import device, note, to_dev

pytestmark = pytest.mark.gpu

W = dict(alpha=2.0, gamma=0.75, delta=5.0, eps=0.25)


def _run(keys, phi, s_hat, heavy, n_mode="device", **w):
    import paper_2607_22578_amd as hs
    dev = device()
    R = keys.shape[0]
    plan = hs.hs_merge_plan(R, 8, 1, 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(max(plan.workspace_bytes, 256), dtype=torch.uint8, device=dev)
    R1 = max(R, 1)
    uk = torch.empty(R1, dtype=torch.int64, device=dev)
    fi = torch.empty(R1, dtype=torch.int32, device=dev)
    ct = torch.empty(R1, dtype=torch.int32, device=dev)
    inv = torch.empty(R1, dtype=torch.int32, device=dev)
    nu = torch.zeros(1, dtype=torch.int64, device=dev)
    st = torch.cuda.current_stream(dev)
    nh = hs.hs_dedup(plan, to_dev(keys), uk, fi, ct, inv, nu, True, ws, stream=st)
    phf = torch.empty(R1, dtype=torch.float64, device=dev)
    pi = torch.empty(R1, dtype=torch.float64, device=dev)
    order = torch.empty(R1, dtype=torch.int32, device=dev)
    hv = to_dev(heavy) if heavy is not None else None
    hs.hs_priority(plan, inv, fi, nh if n_mode == "host" else -1, nu, to_dev(phi), to_dev(s_hat),
                   hv, w["alpha"], w["gamma"], w["delta"], w["eps"], phf, pi, order, ws,
                   stream=st)
    torch.cuda.synchronize(dev)
    return nh, phf[:nh].cpu().numpy(), pi[:nh].cpu().numpy(), order[:nh].cpu().numpy()


def _check(keys, phi, s_hat, heavy, n_mode="device", **w):
    w = dict(W, **w)
    nh, gphi, gpi, gord = _run(keys, phi, s_hat, heavy, n_mode, **w)
    ref = oracle.dedup(keys)
    assert nh == ref["n_unique"]
    rphi, rpi, rord = pr.priorities(ref["inverse"], ref["first_index"], phi, s_hat, heavy,
                                    w["alpha"], w["gamma"], w["delta"], w["eps"])
    np.testing.assert_array_equal(gphi.view(np.uint64), rphi.view(np.uint64))
    np.testing.assert_array_equal(gpi.view(np.uint64), rpi.view(np.uint64))
    np.testing.assert_array_equal(gord, rord)
    return rord


@pytest.mark.parametrize("n_mode", ["device", "host"])
def test_window_priorities(n_mode):
    w = synth.make("ridge1m", with_corpus=False)
    phi, s_hat, heavy = synth.scheduler_inputs(w)
    note(f"priorities on the 1M-row window, n_u from {n_mode}")
    _check(w.keys, phi, s_hat, heavy, n_mode)


def test_many_fused_nodes_merge_passes():
    w = synth.make("dedup256k", with_corpus=False)
    phi, s_hat, heavy = synth.scheduler_inputs(w)
    note("priorities on 262,144 requests")
    _check(w.keys, phi, s_hat, heavy)
    # equal contributions: the order is by group size, then group
    _check(w.keys, np.ones(w.R, np.float32), np.ones(w.R, np.float32), None, alpha=0.0,
           gamma=1.0, delta=0.0, eps=1.0)


@pytest.mark.parametrize("n_u", [1, 2000, 4095, 4096, 4097, 9000])
def test_chunk_boundaries_and_ties(n_u):
    rng = np.random.default_rng(n_u)
    keys = rng.permutation(np.repeat(rng.integers(-2 ** 62, 2 ** 62, size=n_u), 2))
    keys = keys.astype(np.int64)
    R = keys.shape[0]
    phi = rng.choice(np.array([0.0, 1.0, 3.0, 1e9, -2.0, np.nan], np.float32), size=R)
    s_hat = np.full(R, 2.0, np.float32)
    _check(keys, phi, s_hat, None)
    # every priority equal: order = 0 .. n_u-1
    ordr = _check(keys, np.zeros(R, np.float32), s_hat, None)
    assert (ordr == np.arange(len(ordr))).all()
