"""The library's calls captured in a HIP graph (torch.cuda.CUDAGraph) and replayed.

Every entry point only enqueues kernels on the caller's stream: no memset, no
allocation, no host synchronisation.  A captured step therefore replays as the
eager calls would run.  Each replay here runs on new inputs copied in place
between replays, with eager work and a synchronisation in between, and must
equal the eager calls on the same inputs bit for bit (masks, O, LSE)."""
import numpy as np
import pytest

from helpers import small_inputs, stable_seed

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
seer = pytest.importorskip("paper_2410_13276_amd")

REPLAYS = 3


def _bf16(x):
    return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16)


def _capture(step):
    """Warm the step up on a side stream, then capture it (torch's recipe)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def _valid_idx(count, idx):
    """Index-list entries that are defined (the first count[...] of each row)."""
    n = idx.shape[-1]
    keep = torch.arange(n, device=idx.device) < count.unsqueeze(-1).long()
    return torch.where(keep, idx, torch.zeros_like(idx))


@pytest.mark.parametrize("batched", [False, True], ids=["one_launch", "batched_launches"])
def test_gate_sparse_and_dense_attention_replay(batched):
    split = {"split": 1, "split_width": 4}  # the dense call splits its rows into ranges of 4 blocks
    # batched: the sparse call launches its rows in batches of 64 workgroups
    sparse_opts = {"batch_min_blocks": 1, "batch_wgs": 64} if batched else {"batch_min_blocks": -1}
    B, Hq, Hkv, S, D = 1, 8, 2, 4096, 128
    host = [small_inputs(B, Hq, Hkv, S, D, "bf16", seed=stable_seed("graph", r), spikes=True)
            for r in range(REPLAYS)]
    _, q0, k0, v0, wq, wk = host[0]
    qd, kd, vd = (_bf16(x).cuda() for x in (q0, k0, v0))
    wqd, wkd = torch.from_numpy(wq).cuda(), torch.from_numpy(wk).cuda()
    mask = seer.alloc_mask(B, Hq, S, "cuda")
    o_s, o_d, o_u = torch.empty_like(qd), torch.empty_like(qd), torch.empty_like(qd)
    l_s = torch.empty((B, Hq, S), dtype=torch.float32, device="cuda")
    l_d, l_u = torch.empty_like(l_s), torch.empty_like(l_s)
    gws = torch.empty(seer.gate_workspace_bytes(qd, kd, wq.shape[-1]), dtype=torch.uint8, device="cuda")
    aws = torch.empty(max(seer.attn_workspace_bytes(qd, kd, vd, opts=split), 1), dtype=torch.uint8, device="cuda")
    assert aws.numel() > 1, "the dense call should take the key-range split here"

    def step():
        seer.gate(qd, kd, wqd, wkd, mode=seer.TOPK_RATIO, topk_ratio=0.2, mask=mask, workspace=gws)
        seer.bsattn(qd, kd, vd, mask, out=o_s, lse=l_s, opts=sparse_opts)
        seer.dense_attn(qd, kd, vd, out=o_d, lse=l_d, workspace=aws, opts=split)
        seer.dense_attn(qd, kd, vd, out=o_u, lse=l_u)  # unsplit: two query heads per workgroup

    g = _capture(step)
    for r in range(REPLAYS):
        print(f"[graph] replay {r}", flush=True)
        _, q, k, v, _, _ = host[r]
        for dst, src in ((qd, q), (kd, k), (vd, v)):
            dst.copy_(_bf16(src))
        g.replay()
        torch.cuda.synchronize()
        outs = (o_s, l_s, o_d, l_d, o_u, l_u)
        got = [t.clone() for t in (mask.count, _valid_idx(mask.count, mask.idx)) + outs]
        for t in outs:
            t.zero_()
        step()
        torch.cuda.synchronize()
        ref = (mask.count, _valid_idx(mask.count, mask.idx)) + outs
        names = ("count", "idx", "o sparse", "lse sparse", "o split dense", "lse split dense", "o dense",
                 "lse dense")
        for name, a, b in zip(names, got, ref):
            assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"replay {r}: {name} differs"


def test_varlen_replay():
    """Packed variable-length batches launch one batch-1 pass per sequence: the
    launch-bound case a graph exists for."""
    lengths = [300, 64, 1, 2000, 0, 777]
    Hq, Hkv, D = 4, 2, 128
    T = sum(lengths)
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    host = []
    for r in range(REPLAYS):
        _, q, k, v, wq, wk = small_inputs(1, Hq, Hkv, T, D, "bf16", seed=stable_seed("graph-varlen", r), Dg=64)
        host.append([np.ascontiguousarray(x[0].transpose(1, 0, 2)) for x in (q, k, v)] + [wq, wk])
    qd, kd, vd = (_bf16(x).cuda() for x in host[0][:3])
    wqd, wkd = torch.from_numpy(host[0][3]).cuda(), torch.from_numpy(host[0][4]).cuda()
    mask = seer.alloc_varlen_mask(qd, kd, cu)
    out = torch.empty_like(qd)
    lse = torch.empty(Hq * T, dtype=torch.float32, device="cuda")

    def step():
        seer.gate_varlen(qd, kd, wqd, wkd, cu, mode=seer.TOPK_RATIO, topk_ratio=0.3, mask=mask)
        seer.bsattn_varlen(qd, kd, vd, cu, mask, out=out, lse=lse)

    g = _capture(step)
    for r in range(REPLAYS):
        print(f"[graph varlen] replay {r}", flush=True)
        for dst, src in zip((qd, kd, vd), host[r][:3]):
            dst.copy_(_bf16(src))
        g.replay()
        torch.cuda.synchronize()
        got_o, got_l, got_c = out.clone(), lse.clone(), mask.count.clone()
        got_i = [mask.sequence(b)[1].clone() for b in range(len(lengths)) if lengths[b]]
        out.zero_(), lse.zero_()
        step()
        torch.cuda.synchronize()
        assert torch.equal(got_o.view(torch.int16), out.view(torch.int16)), f"replay {r}: O differs"
        assert torch.equal(got_l, lse), f"replay {r}: LSE differs"
        assert torch.equal(got_c, mask.count), f"replay {r}: counts differ"
        ref_i = [mask.sequence(b) for b in range(len(lengths)) if lengths[b]]
        for gi, (c, ri) in zip(got_i, ref_i):
            assert torch.equal(_valid_idx(c, gi), _valid_idx(c, ri)), f"replay {r}: index lists differ"
