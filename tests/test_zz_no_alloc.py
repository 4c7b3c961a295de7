"""cb_pipeline_noalloc (the library's own per-device workspace) against
cb_pipeline (a caller-owned workspace) through the C ABI: bitwise-identical
outputs on two calls in a row, the second on a smaller input, so that the
first call's contents of the shared workspace cannot leak into the second."""
import sys

import numpy as np
import pytest

import cb_workloads as W

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(torch, a):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def test_noalloc_matches_pipeline_on_two_calls():
    import torch

    import paper_2609_32046_amd as cb

    assert torch.cuda.is_available()
    cases = [
        W.custom(layers=4, q_heads=32, kv_heads=8, head_dim=128, q_len=64, seq_len=8192,
                 kdist="chanscale", cfg_id=501),
        W.custom(layers=2, q_heads=8, kv_heads=2, head_dim=64, q_len=16, seq_len=1500,
                 dtype="f32", cfg_id=502),
    ]
    for w in cases:
        say(f"case noalloc L={w.layers} T={w.seq_len} {w.dtype}")
        q = W.gen_q(w)
        K, V = W.gen_kv(w)
        qd, kd, vd = to_dev(torch, q), to_dev(torch, K), to_dev(torch, V)
        lay = cb.layout_of(w)
        ref = cb.Buffers(lay, 0.25)
        got = cb.Buffers(lay, 0.25)
        cb.run_pipeline(qd, kd, vd, ref)
        keep = cb.cb_pipeline_noalloc(qd, kd, vd, lay, 0.25, got.importance, got.idx, got.k_out,
                                      got.v_out, row_lse=got.row_lse)
        torch.cuda.synchronize()
        assert keep == ref.keep
        for name in ("importance", "row_lse", "idx", "k_out", "v_out"):
            a = getattr(ref, name).contiguous().view(-1).view(torch.uint8).cpu().numpy()
            b = getattr(got, name).contiguous().view(-1).view(torch.uint8).cpu().numpy()
            assert a.tobytes() == b.tobytes(), name
