"""The hot path captured in a HIP graph: selector then sparse forward, replayed.

The two C-ABI calls only launch kernels on the caller's stream (no allocation,
no host synchronisation, no memset), so a caller can capture one step and
replay it.  Each replay is checked bit for bit against the eager result, with
other eager work and synchronisations between the replays.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

from synthetic import TINY, generate
from tests.helpers import keep_for, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("split,fused", [(True, False), (False, False), (True, True)],
                         ids=["split", "onepass", "split-fused-selector"])
def test_graph_replay_matches_eager(gpu_lib, split, fused):
    import torch

    S = gpu_lib
    w = TINY.with_(name="graph", head_dim=128, lq=64 * 40 + 9, l_ref=64 * 30 + 3, l_text=150, heads=3, seed=31)
    _say(f"[graph] H={w.heads} D={w.head_dim} Lq={w.lq} Lk={w.lk} split={split} fused={fused}")
    qb, kb, vb = generate(w)
    q, k, v = to_dev(qb), to_dev(kb), to_dev(vb)
    keep, _ = keep_for(S, w)
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    n_q = -(-Lq // w.block)
    stride = S.sparstar_kv_stride(H, Lk, w.block, w.density, keep)
    num = torch.empty((B, H, n_q), dtype=torch.int32, device="cuda")
    idx = torch.empty((B, H, n_q, stride), dtype=torch.int32, device="cuda")
    ws = torch.empty(S.sparstar_score_workspace_bytes(B, H, Lq, Lk, D, w.block), dtype=torch.uint8, device="cuda")
    aws_n = S.sparstar_attn_workspace_bytes(B, H, Lq, Lk, D, w.block)
    aws = torch.empty(max(aws_n, 1), dtype=torch.uint8, device="cuda") if split else None
    o = torch.empty_like(q)
    lse = torch.empty((B, H, Lq), dtype=torch.float32, device="cuda")

    def step():
        S.sparstar_score_blocks(q, k, w.block, w.density, keep, kv_stride=stride, workspace=ws, out=(num, idx),
                                fused=fused)
        S.sparstar_sparse_attn_fwd(q, k, v, num, idx, w.block, out=o, lse=lse, split=split, workspace=aws)

    step()
    torch.cuda.synchronize()
    ref = (num.clone(), idx.clone(), o.clone(), lse.clone())

    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(stream):
        step()  # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=stream):
            step()
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()

    for rep in range(3):
        # clobber the outputs eagerly, then replay
        num.fill_(-7)
        idx.fill_(-7)
        o.zero_()
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        n_ok = torch.equal(num, ref[0])
        idx_ok = all(torch.equal(idx[b, h, i, : int(ref[0][b, h, i])], ref[1][b, h, i, : int(ref[0][b, h, i])])
                     for b in range(B) for h in range(H) for i in range(n_q))
        o_ok = torch.equal(o, ref[2])
        l_ok = torch.equal(lse, ref[3])
        _say(f"[graph] replay {rep}: lists {n_ok and idx_ok}, O {o_ok}, lse {l_ok}")
        assert n_ok and idx_ok and o_ok and l_ok, f"replay {rep} differs from the eager step"
        # unrelated eager work between replays
        x = torch.randn(1 << 20, device="cuda")
        assert np.isfinite(float(x.sum().item()))
