"""Row gather (representative rows, embedding rows of distinct chunk ids,
delivery), bit-exact against the oracle's gather."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_harness import device, note, to_dev

pytestmark = pytest.mark.gpu


def test_chunk_embedding_dedup_and_gather_full_size():
    """1,024 workflows x 256 chunk ids (Zipf 1.0 over 200,000 chunks): distinct
    ids, then their 1024-wide bf16 embedding rows."""
    import paper_2607_22578_amd as hs
    dev = device()
    w = synth.make("dedup256k")
    note(f"dedup256k R={w.R} table={w.table.shape}")
    R = w.R
    plan = hs.hs_merge_plan(R, w.dim, w.table.shape[0], 1, hs.HS_BF16, hs.HS_BF16)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=dev)
    kd = torch.from_numpy(w.keys).to(dev)
    uk = torch.empty(R, dtype=torch.int64, device=dev)
    fi = torch.empty(R, dtype=torch.int32, device=dev)
    ct = torch.empty(R, dtype=torch.int32, device=dev)
    inv = torch.empty(R, dtype=torch.int32, device=dev)
    nu = torch.zeros(1, dtype=torch.int64, device=dev)
    table = to_dev(w.table)
    out = torch.zeros((R, w.dim), dtype=torch.bfloat16, device=dev)
    st = torch.cuda.current_stream(dev)
    hs.hs_dedup(plan, kd, uk, fi, ct, inv, nu, None, ws, stream=st)
    hs.hs_scatter(table, table.shape[0], w.dim * 2, uk, 1, R, nu, out, stream=st)
    torch.cuda.synchronize(dev)
    ref = oracle.dedup(w.keys)
    n = ref["n_unique"]
    assert int(nu.item()) == n
    np.testing.assert_array_equal(uk[:n].cpu().numpy(), ref["unique_keys"])
    np.testing.assert_array_equal(inv.cpu().numpy(), ref["inverse"])
    want = oracle.gather_rows(w.table, ref["unique_keys"])
    got = out[:n].cpu().view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, want)
    # rows past n_unique were not written
    assert torch.count_nonzero(out[n:].view(torch.int16)).item() == 0


@pytest.mark.parametrize("row_bytes,is64", [(40, 0), (12, 1), (48, 0), (4096, 1), (1540, 0)])
def test_gather_rows_widths(row_bytes, is64):
    import paper_2607_22578_amd as hs
    dev = device()
    rng = np.random.default_rng(row_bytes)
    src_rows, n_out = 999, 3001
    src = rng.integers(0, 2 ** 32, size=(src_rows, row_bytes // 4), dtype=np.uint32)
    idx = rng.integers(0, src_rows, size=n_out).astype(np.int64 if is64 else np.int32)
    idx[5] = -1          # out of range: row left unwritten
    idx[6] = src_rows
    sd = torch.from_numpy(src.view(np.int32)).to(dev)
    idd = torch.from_numpy(idx).to(dev)
    dst = torch.full((n_out, row_bytes // 4), -1, dtype=torch.int32, device=dev)
    limit = torch.tensor([n_out - 10], dtype=torch.int64, device=dev)
    hs.hs_scatter(sd, src_rows, row_bytes, idd, is64, n_out, limit, dst)
    torch.cuda.synchronize(dev)
    got = dst.cpu().numpy().view(np.uint32)
    ok = (idx >= 0) & (idx < src_rows)
    ok[n_out - 10:] = False
    want = oracle.gather_rows(src, np.where(ok, idx, 0).astype(idx.dtype))
    np.testing.assert_array_equal(got[ok], want[ok])
    assert np.all(got[~ok] == 0xFFFFFFFF)


def test_deliver_both_arrays_and_workflow_rows():
    """hs_deliver: out[i] = topk[inverse[i]] for scores and indices in one
    launch, bit-exact against the oracle's gather; groups outside the topk
    rows leave their requests untouched; workflow w's requests are the rows
    hs_workflow_rows names."""
    import paper_2607_22578_amd as hs
    dev = device()
    rng = np.random.default_rng(5)
    R, k, rows = 3001, 13, 400
    off = np.concatenate([[0], np.sort(rng.integers(0, R, 6)), [R]]).astype(np.int64)
    plan = hs.hs_merge_plan(R, 8, 1000, k, hs.HS_BF16, hs.HS_BF16, n_workflows=len(off) - 1,
                            workflow_offsets=off)
    ts = rng.standard_normal((rows, k)).astype(np.float32)
    ti = rng.integers(0, 1000, (rows, k)).astype(np.int32)
    inv = rng.integers(0, rows, R).astype(np.int32)
    inv[[3, 77]] = rows          # outside: left unwritten
    inv[100] = -1
    os_ = torch.full((R, k), 0.5, dtype=torch.float32, device=dev)
    oi = torch.full((R, k), -9, dtype=torch.int32, device=dev)
    hs.hs_deliver(plan, to_dev(ts), to_dev(ti), rows, to_dev(inv), os_, oi)
    torch.cuda.synchronize(dev)
    ok = (inv >= 0) & (inv < rows)
    got_s, got_i = os_.cpu().numpy(), oi.cpu().numpy()
    np.testing.assert_array_equal(got_s[ok].view(np.uint32),
                                  oracle.gather_rows(ts, inv[ok]).view(np.uint32))
    np.testing.assert_array_equal(got_i[ok], oracle.gather_rows(ti, inv[ok]))
    assert np.all(got_s[~ok] == 0.5) and np.all(got_i[~ok] == -9)
    for wf in range(len(off) - 1):
        assert hs.hs_workflow_rows(plan, wf) == (int(off[wf]), int(off[wf + 1] - off[wf]))
