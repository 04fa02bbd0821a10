"""Pins of the oracle's node signatures (oracle/signature.py) against facts
fixed outside it: the FIPS 180-4 example digests (and the key read from
them), messages written out by hand from the layout (tests/golden), a table
of normalisation cases, injectivity of the field encoding, predecessor
propagation through a DAG, the clamping and zero-digest rules, and the
synthetic renderings (one key per template)."""
import hashlib
import json
import os

import numpy as np
import pytest

from oracle import signature as sg
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "signature_worked.json")

# FIPS 180-4 example digests (the NIST "abc", empty and two-block messages)
FIPS = [
    (b"abc", "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"),
    (b"", "e3b0c44298fc1c149afbf4c8996fb92427ae41e4649b934ca495991b7852b855"),
    (b"abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq",
     "248d6a61d20638b8e5c026930c3e6039a33ce45964ff2167f6ecedd419db06c1"),
]


@pytest.mark.parametrize("msg,hexd", FIPS)
def test_fips_digests_and_keys(msg, hexd):
    d = hashlib.sha256(msg).digest()
    assert d.hex() == hexd
    # key = first 8 bytes big-endian, two's complement
    top = int(hexd[:16], 16)
    assert sg.key_of(d) == (top - (1 << 64) if top >= 1 << 63 else top)


def test_key_sign_examples():
    assert sg.key_of(bytes.fromhex("ba7816bf8f01cfea") + bytes(24)) == 0xba7816bf8f01cfea - 2 ** 64
    assert sg.key_of(bytes.fromhex("7fffffffffffffff") + bytes(24)) == 2 ** 63 - 1
    assert sg.key_of(bytes(32)) == 0


def test_hand_written_messages():
    doc = json.load(open(GOLDEN))
    for c in doc["cases"]:
        preds = [bytes.fromhex(h) for h in c["preds_hex"]]
        m = sg.message(c["op_type"], bytes.fromhex(c["params_hex"]), c["text"].encode(), preds,
                       c["normalize"])
        assert m.hex() == c["message_hex"], c["what"]
        assert sg.digest(c["op_type"], bytes.fromhex(c["params_hex"]), c["text"].encode(), preds,
                         c["normalize"]) == hashlib.sha256(bytes.fromhex(c["message_hex"])).digest()


@pytest.mark.parametrize("raw,norm", [
    (b"", b""),
    (b" \t\n\r\x0b\x0c ", b""),
    (b"\tA\x0bB\x0c", b"a b"),
    (b"MiXeD   case\r\n", b"mixed case"),
    (b"  lead and trail  ", b"lead and trail"),
    (b"one", b"one"),
    (b"Z@[`{", b"z@[`{"),                         # only A-Z fold
    (b"\xc3\x89T\xc3\xa9", b"\xc3\x89t\xc3\xa9"),  # non-ASCII bytes unchanged
    (b"a\x1cb\x85c", b"a\x1cb\x85c"),              # not ASCII whitespace
    (b"a\x00b", b"a\x00b"),
])
def test_normalisation_table(raw, norm):
    assert sg.normalize(raw) == norm


def test_field_encoding_is_injective():
    base = sg.digest(2, b"ab", b"", ())
    assert sg.digest(2, b"a", b"b", ()) != base            # field boundary moved
    assert sg.digest(3, b"ab", b"", ()) != base            # operator type
    p1, p2 = bytes([1]) * 32, bytes([2]) * 32
    assert sg.digest(2, b"", b"x", (p1, p2)) != sg.digest(2, b"", b"x", (p2, p1))  # order
    assert sg.digest(2, b"", b"x", (p1,)) != sg.digest(2, b"", b"x", ())
    assert sg.digest(2, b"", b"A b", (), True) == sg.digest(2, b"", b"a  B", (), True)
    assert sg.digest(2, b"", b"A b", (), False) != sg.digest(2, b"", b"a  B", (), False)


def _pack(items):
    off = np.zeros(len(items) + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(x) for x in items])
    return b"".join(items), off


def test_dag_propagation_and_rules():
    # level 0: two query nodes; level 1: a retrieval node on each, and one on
    # both; node 5 names a predecessor in its own level (zero digest)
    texts = [b"What is HBM", b"what   is hbm", b"", b"", b"", b""]
    params = [b"", b""] + [b"\x0a\x00\x00\x00"] * 4
    op = np.array([1, 1, 2, 2, 2, 2], dtype=np.uint32)
    preds = [[], [], [0], [1], [0, 1], [4]]
    t, toff = _pack(texts)
    p, poff = _pack(params)
    qoff = np.zeros(7, dtype=np.int32)
    qoff[1:] = np.cumsum([len(x) for x in preds])
    qidx = np.array([u for x in preds for u in x], dtype=np.int32)
    dig, keys = sg.signatures(op, p, poff, t, toff, qoff, qidx, [(0, 2), (2, 4)], True)
    assert keys[0] == keys[1]                       # same normalised text
    assert keys[2] == keys[3]                       # same parent signature
    d0 = dig[0].tobytes()
    assert dig[4].tobytes() == sg.digest(2, params[4], b"", (d0, d0))
    assert dig[5].tobytes() == sg.digest(2, params[5], b"", (bytes(32),))
    # a changed parent changes the child
    texts2 = list(texts)
    texts2[0] = b"what is ddr"
    t2, toff2 = _pack(texts2)
    _, keys2 = sg.signatures(op, p, poff, t2, toff2, qoff, qidx, [(0, 2), (2, 4)], True)
    assert keys2[2] != keys[2] and keys2[3] == keys[3]


def test_offset_clamping():
    text = b"abcdef"
    op = np.array([5, 5, 5], dtype=np.uint32)
    off = np.array([0, 4, 100, 2], dtype=np.int64)    # node 1 runs past the end; node 2 reversed
    dig, _ = sg.signatures(op, b"", None, text, off, None, None, [(0, 3)], False)
    assert dig[0].tobytes() == sg.digest(5, b"", b"abcd", (), False)
    assert dig[1].tobytes() == sg.digest(5, b"", b"ef", (), False)
    assert dig[2].tobytes() == sg.digest(5, b"", b"", (), False)


def test_renderings_share_one_key_per_template():
    w = synth.make("ridge1m", with_corpus=False)
    buf, off = synth.render_texts(w.seed, w.template_ids)
    op = np.full(w.R, 2, dtype=np.uint32)
    _, keys = sg.signatures(op, b"", None, buf.tobytes(), off, None, None, [(0, w.R)], True)
    by_t = {}
    for t, k in zip(w.template_ids, keys):
        assert by_t.setdefault(int(t), int(k)) == int(k)
    assert len(set(by_t.values())) == len(by_t)     # no two templates collide
    _, raw = sg.signatures(op, b"", None, buf.tobytes(), off, None, None, [(0, w.R)], False)
    assert len(np.unique(raw)) > len(by_t)          # unnormalised renderings differ
