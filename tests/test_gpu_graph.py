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
