"""One decode step (lsa_index_decode + paged lsa_sparse_attn) captured into a HIP graph replays to
the eager result: every replay, with eager work clobbering the outputs and synchronisations in
between, must give bit-identical index lists, runs, outputs and LSE. The library's calls launch
kernels only (no allocation, no memset), so they are capturable on the caller's stream."""
from __future__ import annotations

import pytest
import torch

from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def test_decode_step_graph_replays_match_eager():
    w = W.SMALL_DECODE
    dev = torch.device("cuda:0")
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    inp = synth.indexer_inputs(w.seed, w.batch, n_phys * w.kv_page, w.n_heads, w.head_dim, w.fp8)
    prm, aprm = w.index_params(), w.attn_params()
    H, dqk, dv = w.attn_dims
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks)
    a = synth.attention_inputs(w.seed, 0, w.batch, n_phys * w.kv_page, H, dqk, dv, latent=True)
    Q = P.bf16_dev(a["q"])
    KV = P.bf16_dev(a["kv"]).view(n_phys, w.kv_page, dqk)
    ctx_d, table_d = P.to_dev(ctx), P.to_dev(table)
    B = w.batch
    out = dict(idx=torch.empty((B, w.k_cap), dtype=torch.int32, device=dev),
               count=torch.empty((B,), dtype=torch.int32, device=dev),
               runs=torch.empty((B, w.k_cap, 2), dtype=torch.int32, device=dev),
               run_count=torch.empty((B,), dtype=torch.int32, device=dev))
    ws_i = torch.empty(max(1, lsa.index_workspace_size(prm, B, table.shape[1] * w.kv_page)), dtype=torch.uint8,
                       device=dev)
    ws_a = torch.empty(max(1, lsa.attn_workspace_size(aprm, B, w.k_cap, True)), dtype=torch.uint8, device=dev)
    O = torch.empty((B, H, dv), dtype=torch.bfloat16, device=dev)
    L = torch.empty((B, H), dtype=torch.float32, device=dev)

    def step():
        lsa.index_decode(prm, ctx_d, table_d, w.kv_page, n_phys, q, wt, k, ks, bk, runs=True, workspace=ws_i, out=out)
        lsa.sparse_attn(aprm, Q, KV, None, out["idx"], out["count"], page_table=table_d, kv_page_size=w.kv_page,
                        out=O, lse=L, workspace=ws_a)

    step()
    torch.cuda.synchronize()
    ref = {key: v.clone() for key, v in out.items()}
    ref_o, ref_l = O.clone(), L.clone()
    assert int(ref["count"].min()) > 0

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        # eager work between replays: clobber every output
        for v in out.values():
            v.fill_(-7)
        O.fill_(3.0)
        L.fill_(-1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        P.assert_same_index_outputs({k_: v.cpu().numpy() for k_, v in out.items()},
                                    {k_: v.cpu().numpy() for k_, v in ref.items()})
        assert torch.equal(O.view(torch.int16), ref_o.view(torch.int16)), rep
        assert torch.equal(L, ref_l), rep
