"""Node signatures on the device (hs_signature) against the oracle, digests
and keys bit-exact: the 1M-row workload's request texts (normalised and raw),
every text length across the SHA-256 padding boundaries, long multi-block
texts at unaligned offsets, a text that ends at a buffer end that is not a
multiple of 16, a three-level DAG hashed level by level, the clamping and
zero-digest rules, a sub-range call, and the whole path fed by the device
keys."""
import numpy as np
import pytest
import torch

import oracle
from oracle import signature as sg
import synth
from gpu_harness import device, note, to_dev

pytestmark = pytest.mark.gpu


def _dev_bytes(b: bytes, pad: int = 0):
    a = np.frombuffer(bytes(b) + bytes(pad), dtype=np.uint8).copy()
    if a.size == 0:
        a = np.zeros(1, dtype=np.uint8)
    return torch.from_numpy(a).to(device())


def _gpu_sig(op, params, poff, text, toff, qoff, qidx, levels, normalize, text_bytes=None,
             keys=True, init=None):
    import paper_2607_22578_amd as hs
    dev = device()
    n = len(op)
    opd = torch.from_numpy(np.asarray(op, dtype=np.uint32).view(np.int32)).to(dev)
    pd = _dev_bytes(params) if params is not None else None
    td = _dev_bytes(text) if text is not None else None
    pod = torch.from_numpy(np.asarray(poff, dtype=np.int64)).to(dev) if poff is not None else None
    tod = torch.from_numpy(np.asarray(toff, dtype=np.int64)).to(dev) if toff is not None else None
    qod = torch.from_numpy(np.asarray(qoff, dtype=np.int32)).to(dev) if qoff is not None else None
    qid = (torch.from_numpy(np.asarray(qidx, dtype=np.int32)).to(dev)
           if qidx is not None and len(qidx) else None)
    dig = torch.zeros((max(n, 1), 32), dtype=torch.uint8, device=dev)
    if init is not None:
        dig.copy_(torch.from_numpy(init))
    kd = torch.zeros(max(n, 1), dtype=torch.int64, device=dev) if keys else None
    st = torch.cuda.current_stream(dev)
    for first, count in levels:
        hs.hs_signature(opd, n, first, count, dig, kd, params=pd, param_off=pod,
                        param_bytes=len(params) if params is not None else 0, text=td,
                        text_off=tod, text_bytes=len(text) if text_bytes is None else text_bytes,
                        pred_off=qod, pred_idx=qid,
                        pred_count=0 if qid is None else len(qidx),
                        flags=hs.HS_SIG_NORMALIZE_TEXT if normalize else 0, stream=st)
    torch.cuda.synchronize(dev)
    return dig[:n].cpu().numpy(), (kd[:n].cpu().numpy() if keys else None)


def _check(op, params, poff, text, toff, qoff, qidx, levels, normalize, **kw):
    gd, gk = _gpu_sig(op, params, poff, text, toff, qoff, qidx, levels, normalize, **kw)
    rd, rk = sg.signatures(op, params or b"", poff, text or b"", toff, qoff, qidx, levels,
                           normalize)
    if kw.get("init") is not None:
        done = np.zeros(len(op), dtype=bool)
        for f, c in levels:
            done[f:f + c] = True
        rd[~done] = kw["init"][~done]
    bad = np.nonzero((gd != rd).any(axis=1))[0]
    assert bad.size == 0, f"{bad.size} digests differ, first node {bad[:5]}"
    if gk is not None:
        sel = np.zeros(len(op), dtype=bool)
        for f, c in levels:
            sel[f:f + c] = True
        np.testing.assert_array_equal(gk[sel], rk[sel])
    return gd, gk


def _pack(items):
    off = np.zeros(len(items) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in items])
    return b"".join(items), off


@pytest.mark.parametrize("normalize", [True, False])
def test_workload_texts(normalize):
    w = synth.make("ridge1m", with_corpus=False)
    buf, off = synth.render_texts(w.seed, w.template_ids)
    note(f"signatures of {w.R} request texts, normalize={normalize}")
    op = np.full(w.R, 2, dtype=np.uint32)
    par = np.full(w.R, 10, dtype=np.uint32).tobytes()            # Top-K per node
    poff = np.arange(w.R + 1, dtype=np.int64) * 4
    _check(op, par, poff, buf.tobytes(), off, None, None, [(0, w.R)], normalize)


def test_every_length_across_padding_boundaries():
    # message length 16 + P + D: P = 4, D = 0..300 crosses 55/56/63/64 mod 64
    rng = np.random.default_rng(3)
    texts = [bytes(rng.integers(33, 127, size=D, dtype=np.uint8)) for D in range(301)]
    t, toff = _pack(texts)
    n = len(texts)
    op = rng.integers(0, 2 ** 32, size=n, dtype=np.uint64).astype(np.uint32)
    par = np.arange(n, dtype=np.uint32).tobytes()
    poff = np.arange(n + 1, dtype=np.int64) * 4
    _check(op, par, poff, t, toff, None, None, [(0, n)], False)
    _check(op, par, poff, t, toff, None, None, [(0, n)], True)


def test_whitespace_heavy_texts_and_params():
    rng = np.random.default_rng(4)
    alphabet = np.frombuffer(b" \t\n\r\x0b\x0cAbZz\xc3\x89\x00\x1c.", dtype=np.uint8)
    texts = [bytes(alphabet[rng.integers(0, len(alphabet), size=int(rng.integers(0, 90)))])
             for _ in range(700)]
    params = [bytes(rng.integers(0, 256, size=int(rng.integers(0, 41)), dtype=np.uint8))
              for _ in range(700)]
    t, toff = _pack(texts)
    p, poff = _pack(params)
    op = np.full(700, 3, dtype=np.uint32)
    _check(op, p, poff, t, toff, None, None, [(0, 700)], True)


def test_long_texts_unaligned_and_buffer_tail():
    rng = np.random.default_rng(5)
    lens = [5000, 1, 777, 4097, 0, 3333, 61]
    texts = [bytes(rng.integers(0, 256, size=L, dtype=np.uint8)) for L in lens]
    t, toff = _pack([b"xyz"] + texts)   # shifted: no text starts 16-aligned
    toff = toff[1:]
    assert len(t) % 16 != 0             # the last text ends inside a partial 16-byte block
    op = np.arange(len(lens), dtype=np.uint32)
    _check(op, None, None, t, toff, None, None, [(0, len(lens))], False)
    _check(op, None, None, t, toff, None, None, [(0, len(lens))], True)


def test_dag_level_by_level():
    rng = np.random.default_rng(6)
    sizes = [300, 200, 100]
    n = sum(sizes)
    texts = [bytes(rng.integers(97, 123, size=int(rng.integers(0, 120)), dtype=np.uint8))
             for _ in range(n)]
    preds, qoff = [], [0]
    base = 0
    levels = []
    for L, sz in enumerate(sizes):
        for v in range(base, base + sz):
            m = 0 if L == 0 else int(rng.integers(0, 5))
            preds += [int(u) for u in rng.integers(0, base, size=m)] if m else []
            qoff.append(len(preds))
        levels.append((base, sz))
        base += sz
    # rule cases: a predecessor inside its own level, a negative id, one past the end
    preds[-1], preds[-2], preds[-3] = n - 1, -7, 10 ** 6
    t, toff = _pack(texts)
    op = rng.integers(0, 9, size=n).astype(np.uint32)
    note(f"DAG of {n} nodes, {len(preds)} edges, 3 levels")
    _check(op, None, None, t, toff, np.array(qoff, dtype=np.int32),
           np.array(preds, dtype=np.int32), levels, True)


def test_clamped_offsets_and_subrange():
    text = b"The Quick Brown Fox Jumps"
    toff = np.array([0, 4, 100, 2, -5, 9, 9, 25], dtype=np.int64)
    op = np.full(7, 1, dtype=np.uint32)
    init = np.random.default_rng(8).integers(0, 256, size=(7, 32), dtype=np.uint8)
    _check(op, None, None, text, toff, None, None, [(0, 7)], True)
    # only nodes [2, 5): the others keep their rows
    _check(op, None, None, text, toff, None, None, [(2, 3)], True, init=init)
    _gpu_sig(op, None, None, text, toff, None, None, [(0, 7)], True, keys=False)


def test_whole_path_on_device_keys():
    import paper_2607_22578_amd as hs
    from gpu_harness import check_unique_topk, check_delivery
    dev = device()
    w = synth.make("ridge1m", n_corpus=5000)
    buf, off = synth.render_texts(w.seed, w.template_ids)
    op = np.full(w.R, 2, dtype=np.uint32)
    _, gk = _check(op, None, None, buf.tobytes(), off, None, None, [(0, w.R)], True)
    m = hs.MergedRetrieval(w.R, w.dim, 5000, w.k, hs.HS_BF16, hs.HS_BF16, device=dev)
    qd, cd = to_dev(w.q_req), to_dev(w.corpus)
    kd = torch.from_numpy(gk).to(dev)
    m.run(kd, qd, cd, stream=torch.cuda.current_stream(dev))
    torch.cuda.synchronize(dev)
    ref = oracle.dedup(gk)
    assert int(m.n_unique.item()) == ref["n_unique"] == len(np.unique(w.template_ids))
    np.testing.assert_array_equal(m.first_index[:ref["n_unique"]].cpu().numpy(),
                                  ref["first_index"])
    check_unique_topk(m, ref, w.q_req, w.corpus, w.k)
    check_delivery(m, w.R)


def test_group_text_beyond_the_lds_copy():
    # 60 texts of ~2 KB in one group of nodes: the group's text range exceeds
    # the bytes it copies to LDS, so later nodes read global memory
    rng = np.random.default_rng(9)
    alphabet = np.frombuffer(b"  \tAbcXyz\n", dtype=np.uint8)
    texts = [bytes(alphabet[rng.integers(0, len(alphabet), size=int(rng.integers(1500, 2600)))])
             for _ in range(60)]
    t, toff = _pack(texts)
    assert len(t) > 48 * 1024
    op = np.full(60, 4, dtype=np.uint32)
    _check(op, None, None, t, toff, None, None, [(0, 60)], True)
    _check(op, None, None, t, toff, None, None, [(0, 60)], False)


def test_long_parameters_and_digests_across_rounds():
    # parameter blobs longer than a 192-byte round, texts around a round,
    # and up to 9 predecessor digests, so that every field of the message
    # can straddle a round boundary
    rng = np.random.default_rng(12)
    n0, n1 = 50, 150
    n = n0 + n1
    params = [bytes(rng.integers(0, 256, size=int(rng.integers(0, 700)), dtype=np.uint8))
              for _ in range(n)]
    texts = [bytes(rng.choice(np.frombuffer(b"aB \t\nxyZ", np.uint8),
                              size=int(rng.integers(0, 400)))) for _ in range(n)]
    preds, qoff = [], [0]
    for v in range(n):
        if v >= n0:
            preds += [int(u) for u in rng.integers(0, n0, size=int(rng.integers(0, 10)))]
        qoff.append(len(preds))
    p, poff = _pack(params)
    t, toff = _pack(texts)
    op = rng.integers(0, 50, size=n).astype(np.uint32)
    for norm in (True, False):
        _check(op, p, poff, t, toff, np.array(qoff, np.int32), np.array(preds, np.int32),
               [(0, n0), (n0, n1)], norm)
