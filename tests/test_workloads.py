"""Seeded generators: deterministic, of the configured shapes, and the same
bytes on every device (no GPU needed for the CPU side)."""
import numpy as np
import pytest
import torch

from paper_2608_25431_amd import workloads as W


def check_table(t):
    segs = t.segs
    order = np.argsort(segs["row_begin"])
    end = 0
    for i in order:
        assert segs[i]["row_begin"] >= end and segs[i]["row_count"] >= 1
        end = segs[i]["row_begin"] + segs[i]["row_count"]
    assert end <= t.n_rows


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_deterministic_and_well_formed(name):
    a, b = W.get(name), W.get(name)
    assert a.keys.tobytes() == b.keys.tobytes() and a.nonce_base.tobytes() == b.nonce_base.tobytes()
    for ta, tb in zip(a.tensors, b.tensors):
        assert ta.segs.tobytes() == tb.segs.tobytes()
        check_table(ta)
        pairs = {(int(s["user"]), int(s["iv_seq"])) for s in ta.segs}
        assert len(pairs) == len(ta.segs)
    # (user, iv_seq) never repeats across the tensors of one workload
    allp = [(int(s["user"]), int(s["iv_seq"])) for t in a.tensors for s in t.segs]
    assert len(set(allp)) == len(allp)


def test_shapes():
    t = W.tiny().tensors[0]
    assert (t.n_rows, t.row_bytes, len(t.segs)) == (16, 8192, 4) and t.segs["row_count"].sum() == 16
    w = W.llama3_8b_kv()
    t = w.tensors[0]
    assert t.row_bytes == 65536 and len(t.segs) == 64 and w.n_users == 16
    assert all(s["row_count"] % 32 == 0 and 8 * 32 <= s["row_count"] <= 128 * 32 for s in t.segs)
    w = W.tamper()
    assert len(w.tensors[0].segs) == 128 and w.n_users == 32
    assert len(w.tamper) == 2 and {k for (_, _, k, _, _) in w.tamper} == {"ct", "tag"}
    assert len(w.mixed) == 2
    assert not {i for (_, i, _, _, _) in w.tamper} & {i for (_, i, _, _) in w.mixed}
    w = W.decode_batch()
    h, tok = w.tensors
    assert h.row_bytes == 16384 and tok.row_bytes == 4 and len(h.segs) == 1024
    assert all(1 <= s["row_count"] <= 4 for s in h.segs)
    assert (h.segs["row_begin"] == tok.segs["row_begin"]).all()
    w = W.llama3_70b_kv()
    t = w.tensors[0]
    assert w.in_place and t.labels is not None and len(t.segs) == 32 and w.n_users == 8
    assert all(128 * 80 <= s["row_count"] <= 512 * 80 for s in t.segs)


def test_data_generator_is_counter_based():
    t = W.tiny().tensors[0]
    full = t.generate("cpu")
    part = t.generate("cpu", 4096, 512)
    assert torch.equal(full[4096:4608], part)
    v = full.view(torch.bfloat16).float()
    assert abs(v.mean().item()) < 0.05 and abs(v.std().item() - 1.0) < 0.05
    tok = W.decode_batch().tensors[1].generate("cpu").view(torch.int32)
    assert int(tok.min()) >= 0 and int(tok.max()) < W.VOCAB
