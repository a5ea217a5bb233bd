"""Graph capture of the resident lookup + inject path: a decode loop of
tfe_lookup_inject calls captured once into a HIP graph (through torch's
CUDA-graph API) and replayed.  Every replay, with eager work and
synchronisation between replays, must reproduce the eager outputs byte for
byte."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu


def test_captured_decode_steps_replay_exactly():
    table = synth.config2_table()
    gt = H.GpuTable(table)
    steps = 8
    batches = [synth.decode_batch(1, 64, set_index=300 + k) for k in range(steps)]
    toks = [torch.from_numpy(b.tokens).cuda() for b in batches]
    hids = [H.to_device(b.hidden(), synth.BF16) for b in batches]
    outs = [H.Outputs(64, 1024, synth.BF16) for _ in range(steps)]

    def loop():
        s = torch.cuda.current_stream().cuda_stream
        for k in range(steps):
            tfe.tfe_lookup_inject(gt.handle, toks[k], 64, 2, 1, hids[k], outs[k].out, outs[k].hit,
                                  outs[k].slot, outs[k].len, tfe.TFE_GATE_SIGMOID, 1.0, s)

    loop()
    torch.cuda.synchronize()
    want = [(o.out.cpu().clone(), o.hit.cpu().clone(), o.slot.cpu().clone()) for o in outs]

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        loop()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        loop()
    for rep in range(3):
        for o in outs:  # eager work between replays
            o.out.fill_(0)
            o.hit.fill_(0xEE)
            o.slot.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, (wo, wh, ws) in zip(outs, want):
            assert torch.equal(o.out.cpu().view(torch.int16), wo.view(torch.int16)), rep
            assert torch.equal(o.hit.cpu(), wh) and torch.equal(o.slot.cpu(), ws)
    del g
    gt.close()


def test_calls_with_host_state_refuse_capture():
    """Lookups on tiered tables, prefetch and n-gram construction keep
    per-call host state or synchronise: on a capturing stream they return
    TFE_ERR_UNSUPPORTED and enqueue nothing, while a resident lookup in the
    same capture is recorded and replays correctly; the tiered table still
    works eagerly afterwards."""
    from .test_gpu_tiered import TieredTable
    table, batch = synth.config1()
    res = H.GpuTable(table)
    tier = TieredTable(table, 32, 0, adopt=False)
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), table.dtype)
    o_res, o_tier = H.Outputs(batch.T, table.dim, table.dtype), H.Outputs(batch.T, table.dim,
                                                                          table.dtype)
    tail = tok[:, -2:].contiguous()
    cand = torch.zeros((batch.B, 2), dtype=torch.int32, device="cuda")
    tup = torch.zeros((8, 2), dtype=torch.int32, device="cuda")
    cnt = torch.zeros(8, dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    statuses = []
    with torch.cuda.graph(g):
        s = torch.cuda.current_stream().cuda_stream
        H.run(res, tok, batch.B, batch.ctx, batch.S, h, o_res, stream=s)
        calls = [
            lambda: tfe.tfe_lookup_inject(tier.handle, tok, batch.B, batch.ctx, batch.S, h,
                                          o_tier.out, o_tier.hit, o_tier.slot, o_tier.len,
                                          tfe.TFE_GATE_SIGMOID, 1.0, s),
            lambda: tfe.tfe_prefetch(tier.handle, tail, 2, cand, batch.B, 2, s),
            lambda: tfe.tfe_ngram_top(tok, tok.numel(), synth.V, 2, 0, 8, tup, cnt, s),
        ]
        for call in calls:
            try:
                call()
                statuses.append(0)
            except tfe.TfeError as e:
                statuses.append(e.status)
    assert statuses == [tfe.TFE_ERR_UNSUPPORTED] * 3
    assert tfe.tfe_get_stats(tier.handle)["calls"] == 0  # refused before counting
    o_res.out.fill_(0)
    o_res.slot.fill_(-7)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    hit, row, ln, want = H.oracle_answer(table, H.oracle_table(table), batch.tokens, batch.ctx,
                                         batch.S, batch.hidden())
    np.testing.assert_array_equal(o_res.slot.cpu().numpy(), row)
    H.assert_close(H.to_host(o_res.out, table.dtype), want, table.dtype)
    tfe.tfe_lookup_inject(tier.handle, tok, batch.B, batch.ctx, batch.S, h, o_tier.out,
                          o_tier.hit, o_tier.slot, o_tier.len, tfe.TFE_GATE_SIGMOID, 1.0,
                          H.cur_stream())
    torch.cuda.synchronize()
    assert tfe.tfe_get_stats(tier.handle)["calls"] == 1
    np.testing.assert_array_equal(o_tier.slot.cpu().numpy(), row)
    H.assert_close(H.to_host(o_tier.out, table.dtype), want, table.dtype)
    del g
    tier.close()
    res.close()
