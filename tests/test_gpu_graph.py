"""The whole window (dedup, representative rows, score and top-k, merge,
delivery) captured once as a HIP graph and replayed on windows whose
contents change between replays: every replay equals the eager path on the
same window bit for bit.  Between replays the program runs its own eager
window and synchronises; each replay is checked before the next window is
written.  The window issues kernel launches only (the distinct count stays
on the device), which is what makes it capturable."""
import numpy as np
import pytest
import torch

import paper_2607_22578_amd as hs
import synth
from gpu_harness import device, note

pytestmark = pytest.mark.gpu

OUTS = ("unique_keys", "first_index", "counts", "inverse", "n_unique", "topk_score",
        "topk_index", "out_score", "out_index")


def _to_dev(a, dev):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


@pytest.mark.parametrize("enc,tiled", [("bf16", False), ("fp8", False), ("bf16", True)])
def test_window_graph_replays_match_eager(enc, tiled):
    dev = device()
    wins = synth.window_stream("ridge1m", 4)
    w0 = wins[0]
    d, k = w0.dim, w0.k
    n_corpus = 60_000
    c, sc = synth.gaussian_rows(w0.seed, synth.S_CORPUS, n_corpus, d, enc)
    corpus, scale = _to_dev(c, dev), (_to_dev(sc, dev) if sc is not None else None)
    cdt = hs.HS_FP8_E4M3 if enc == "fp8" else hs.HS_BF16
    m = hs.MergedRetrieval(w0.R, d, n_corpus, k, hs.HS_BF16, cdt, device=dev, tiled_corpus=tiled)
    if tiled:   # (made once, outside the captured window)
        corpus = m.tile_corpus(corpus)
        torch.cuda.synchronize(dev)
    keys = _to_dev(wins[0].keys, dev).clone()
    q_req = _to_dev(wins[0].q_req, dev).clone()
    s = torch.cuda.Stream(dev)   # default priority
    m.run(keys, q_req, corpus, scale, stream=s)   # warm-up (eager)
    torch.cuda.synchronize(dev)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        m.run(keys, q_req, corpus, scale, stream=s)
    torch.cuda.synchronize(dev)
    note(f"{enc}: window captured (R={w0.R}, N={n_corpus}, k={k})")
    for i in (1, 2, 0, 3):
        keys.copy_(_to_dev(wins[i].keys, dev))
        q_req.copy_(_to_dev(wins[i].q_req, dev))
        torch.cuda.synchronize(dev)
        m.run(keys, q_req, corpus, scale, stream=s)   # eager, the expected result
        torch.cuda.synchronize(dev)
        want = {o: getattr(m, o).clone() for o in OUTS}
        for o in OUTS:   # so that a replay that writes nothing cannot pass
            getattr(m, o).fill_(-1)
        torch.cuda.synchronize(dev)
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize(dev)
        nu = int(want["n_unique"].item())
        assert int(m.n_unique.item()) == nu
        for o in OUTS:
            got, exp = getattr(m, o), want[o]
            rows = w0.R if o in ("inverse", "out_score", "out_index") else nu
            if got.dim() == 1 and got.numel() == 1:
                rows = 1
            assert torch.equal(got[:rows], exp[:rows]), (i, o)
        note(f"{enc}: window {i} replay equals eager (n_u={nu})")
