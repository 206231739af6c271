"""The library under HIP graph capture: one step (head with argmax, block draw, verification)
captured once and replayed, every replay bit-identical to the eager step.

The entry points allocate nothing, synchronise nothing and need no workspace clearing, so a
caller may capture them; between replays the outputs are overwritten by eager work, so each
replay must rewrite all of them.
"""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def test_step_graph_replays_match_eager():
    from paper_2608_05448_amd import dblast as D
    dev = torch.device("cuda:0")
    B, K, R, d, V = 4, 8, 4, 256, 5000
    print(f"[graph] B={B} K={K} R={R} d={d} V={V}", flush=True)
    h = synth.make_uniform_logits((B, K, R, d), 71).to(torch.bfloat16).to(dev)
    w = (synth.make_uniform_logits((V, d), 72) * 0.05).to(torch.bfloat16).to(dev)
    ell = synth.make_uniform_logits((B, R), 73).float().to(dev)
    logp = torch.log_softmax(synth.make_uniform_logits((B, K + 1, V), 74, scale=3.0).double(),
                             dim=-1).float().to(dev)
    nT = D.ntiles(V)
    tls = torch.empty((B, K, R, V), dtype=torch.float32, device=dev)
    lmass = torch.empty((B, K, R, nT), dtype=torch.float32, device=dev)
    lse = torch.empty((B, K, R), dtype=torch.float32, device=dev)
    am = torch.empty((B, K, R), dtype=torch.int32, device=dev)
    z = torch.empty(B, dtype=torch.int32, device=dev)
    x = torch.empty((B, K), dtype=torch.int32, device=dev)
    out = {"n_accept": torch.empty(B, dtype=torch.int32, device=dev),
           "next_token": torch.empty(B, dtype=torch.int32, device=dev),
           "accept_mass": torch.empty((B, K), dtype=torch.float32, device=dev),
           "al_expected": torch.empty(B, dtype=torch.float32, device=dev),
           "exp_len": torch.empty(B, dtype=torch.float32, device=dev)}
    ws_h = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_HEAD, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    ws_s = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_SAMPLE, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    ws_v = torch.empty(D.dbl_workspace_bytes(D.DBL_OP_VERIFY, B, K, R, d, V), dtype=torch.uint8,
                       device=dev)
    results = [tls, lmass, lse, am, z, x] + list(out.values())

    def step():
        D.dbl_head_logprobs(h, w, tls, lmass, lse, argmax=am, ws=ws_h)
        D.dbl_sample_block(tls, lmass, lse, ell, z_temp=1.0, seed=5, step=3, z_out=z, x_out=x,
                           ws=ws_s)
        D.dbl_verify_block(tls, lmass, lse, ell, x, logp, z_temp=1.0, seed=5, step=3, out=out,
                           ws=ws_v)

    step()
    torch.cuda.synchronize()
    eager = [t.clone() for t in results]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on a side stream, as capture requires
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in results:  # eager work between replays: every output overwritten
            t.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got, ref in zip(["tls", "lmass", "lse", "argmax", "z", "x"] + list(out),
                                  results, eager):
            assert torch.equal(got, ref), f"replay {rep}: {name} differs from the eager step"
        print(f"[graph] replay {rep} identical", flush=True)
