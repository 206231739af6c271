"""Full-size GPU runs of the benchmark-scale workloads.

Each test runs the whole hot path at the workload's real shape in the same launch
configuration as the benchmark, then recomputes blocks end to end with the oracle (binary64
head on the same bf16 inputs, then the oracle's own draw and verification): every block of the
Qwen3-8B step at every target temperature and of the Qwen3-4B step, sampled blocks and steps of the objective and stress
workloads. Token
indices must agree exactly; any disagreement must be a certified near-tie (the GPU's fp32
log-probs differ from the oracle's binary64 ones by ~1e-6, which can move a threshold across a
boundary only when it lies within that margin). Real-valued outputs agree within 1e-4 relative.
"""
import numpy as np
import pytest
import torch

import synth
from cases import np32
from oracle import contract as C
from oracle import head as OH
from oracle import mixture as MX

pytestmark = pytest.mark.gpu


def _oracle_factored(h_block, w_np):
    """Oracle branch log-probs of one block's hidden states, in the two-level form
    (tls [K, R, V], lmass [K, R, nT], lse [K, R]) and flat (lq [K, R, V]), binary32."""
    K, R, d = h_block.shape
    tls, lm, ls = OH.head_factored(np32(h_block).reshape(K * R, d), w_np, v_chunk=8192)
    lq = OH.flat_logq(tls, lm, ls).reshape(K, R, -1)
    return tls.reshape(K, R, -1), lm.reshape(K, R, -1), ls.reshape(K, R), lq


def _oracle_lq(h_block, w_np):
    """Oracle branch log-probs [K, R, V] (binary32 flat form) for one block's hidden states."""
    return _oracle_factored(h_block, w_np)[3]


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    m = np.abs(b) > 1e-30
    return float(np.max(np.abs(a[m] - b[m]) / np.abs(b[m]))) if m.any() else 0.0


def _near_tie(weights, r, got, want):
    """True if an inverse CDF on integer `weights` with word r picks `got` instead of `want`
    only because its threshold sits within a relative 1e-5 of the cumulative boundary between
    them."""
    cum = np.cumsum(np.asarray(weights).astype(np.float64))
    Z = cum[-1]
    T = (int(r) * int(Z)) >> 32
    lo, hi = min(got, want), max(got, want)
    gap = min(abs(T - cum[lo]), abs(T - (cum[hi - 1] if hi > 0 else 0.0)))
    return gap <= 1e-5 * Z


def _near_tie_token(tls_row, lm_row, ls, r_tile, r_id, got, want):
    """The two-stage draw of a token: a near-tie in the tile stage when the tiles differ, else
    in the id stage within their common tile."""
    tg, tw = got // MX.TILE, want // MX.TILE
    if tg != tw:
        off = (np.asarray(lm_row, np.float32) - np.float32(ls)).astype(np.float32)
        return _near_tie(C.quant40(C.detexp32(off)), r_tile, tg, tw)
    ids = np.asarray(tls_row[tw * MX.TILE:(tw + 1) * MX.TILE], np.float32)
    return _near_tie(C.quant40(C.detexp32(ids)), r_id, got % MX.TILE, want % MX.TILE)


@pytest.mark.parametrize("name,temps", [("qwen3_8b", synth.QWEN3_8B_TEMPERATURES),
                                        ("qwen3_4b", (synth.WORKLOADS["qwen3_4b"].temperature,))])
def test_e2e_all_blocks(name, temps):
    """The benchmark's step at the Qwen3-8B shape (every target temperature) and the Qwen3-4B
    shape (its own), every block: the oracle's binary64 head on the same bf16 inputs, then its own
    draw and verification."""
    from cases import oracle_full_factored, oracle_full_head
    from paper_2608_05448_amd import dblast as D
    wl = synth.WORKLOADS[name]
    print(f"[fullsize] {name} e2e B={wl.B} K={wl.K} R={wl.R} d={wl.d} V={wl.V}", flush=True)
    h = synth.make_h(wl, "cuda")
    w = synth.make_w(wl, "cuda")
    ell = synth.make_ell(wl, "cuda")
    tls, lmass, lse = D.dbl_head_logprobs(h, w)
    z, x = D.dbl_sample_block(tls, lmass, lse, ell, z_temp=wl.z_temp, seed=wl.philox_seed, step=0)
    torch.cuda.synchronize()
    B, K, R, V = wl.B, wl.K, wl.R, wl.V
    print(f"[fullsize] {name}: oracle head on all {wl.M} rows", flush=True)
    lq_all = oracle_full_head(name, h, w).reshape(B, K, R, V)
    o_tls, o_lm, o_ls = oracle_full_factored(name, h, w)
    o_tls, o_lm, o_ls = o_tls.reshape(B, K, R, V), o_lm.reshape(B, K, R, -1), o_ls.reshape(B, K, R)
    z_g, x_g = z.cpu().numpy(), x.cpu().numpy()
    ell_np = ell.cpu().numpy()
    z_o, x_o = MX.sample_blocks(o_tls, o_lm, o_ls, ell_np, wl.z_temp, wl.philox_seed, 0,
                                np.arange(B))
    np.testing.assert_array_equal(z_g, z_o)
    mismatches = 0
    for b in range(B):
        for k in range(K):
            if x_g[b, k] != x_o[b, k]:
                r0 = C.draw_u32(wl.philox_seed, C.PURPOSE_TOKEN, k, b, 0)
                r1 = C.draw_u32_word1(wl.philox_seed, C.PURPOSE_TOKEN, k, b, 0)
                zb = z_o[b]
                assert _near_tie_token(o_tls[b, k, zb], o_lm[b, k, zb], o_ls[b, k, zb], r0, r1,
                                       x_g[b, k], x_o[b, k])
                mismatches += 1
    print(f"[fullsize] {name} draw: certified near-ties {mismatches}", flush=True)
    # Verification is compared where both sides drafted the same block (all of them unless a
    # certified near-tie moved a token); each side verifies its own draft.
    same = [b for b in range(B) if np.array_equal(x_g[b], x_o[b])]
    assert len(same) >= B - mismatches
    sel = np.array(same)
    for T in temps:
        logp = synth.make_logp(wl, rows=wl.K + 1, device="cuda", temperature=T)
        out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, z_temp=wl.z_temp,
                                 seed=wl.philox_seed, step=0)
        torch.cuda.synchronize()
        lp = logp.cpu().numpy()
        ref = MX.verify_blocks(lq_all[sel], ell_np[sel], wl.z_temp, x_o[sel], lp[sel],
                               wl.philox_seed, 0, sel)
        np.testing.assert_array_equal(out["n_accept"].cpu().numpy()[sel], ref["n_accept"])
        np.testing.assert_array_equal(out["next_token"].cpu().numpy()[sel], ref["next_token"])
        assert _rel(out["accept_mass"].cpu().numpy()[sel], ref["beta"]) < 1e-4
        assert _rel(out["exp_len"].cpu().numpy()[sel], ref["E"]) < 1e-4
        assert _rel(out["al_expected"].cpu().numpy()[sel], ref["al"]) < 1e-4
        na = out["n_accept"].float().mean().item()
        print(f"[fullsize] {name} T={T}: {len(same)} blocks match; mean n_accept {na:.3f}, "
              f"mean E {out['exp_len'].mean().item():.4f}", flush=True)


def test_objective_workload_chunked_expected_length():
    """2048 blocks x K=16 x R=16 at d=4096: chunks of 128 blocks through the head, the
    expected-length reduction and the training-objective forward along target trajectories."""
    from oracle import objective as OB
    from paper_2608_05448_amd import dblast as D
    wl = synth.WORKLOADS["objective"]
    chunk = 128
    print(f"[fullsize] objective {wl.B} blocks K={wl.K} R={wl.R} in chunks of {chunk}", flush=True)
    w = synth.make_w(wl, "cuda")
    ell = synth.make_ell(wl, "cuda")
    beta_all = torch.empty((wl.B, wl.K), dtype=torch.float32, device="cuda")
    e_all = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    j_all = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    lt_all = torch.empty(wl.B, dtype=torch.int32, device="cuda")
    nll_all = torch.empty(wl.B, dtype=torch.float32, device="cuda")
    check = {5: None, 1500: None, 2047: None}
    for c0 in range(0, wl.B, chunk):
        blocks = range(c0, c0 + chunk)
        h = synth.make_h(wl, "cuda", blocks=blocks)
        logp = synth.make_logp(wl, rows=wl.K, device="cuda", blocks=blocks)
        xs = synth.make_trajectory(wl, logp, blocks=blocks)
        tls, lmass, lse = D.dbl_head_logprobs(h, w)
        beta, e = D.dbl_expected_len(tls, lmass, lse, ell[c0:c0 + chunk].contiguous(), xs, logp,
                                     z_temp=wl.z_temp)
        beta_all[c0:c0 + chunk] = beta
        e_all[c0:c0 + chunk] = e
        obj = D.dbl_acceptance_objective(tls, lmass, lse, ell[c0:c0 + chunk].contiguous(), xs,
                                         logp, z_temp=wl.z_temp, tau=0.1, want_terms=False)
        j_all[c0:c0 + chunk] = obj["J"]
        lt_all[c0:c0 + chunk] = obj["ell_tau"]
        nll_all[c0:c0 + chunk] = obj["nll"]
        for b in check:
            if c0 <= b < c0 + chunk:
                i = b - c0
                check[b] = (h[i].clone(), logp[i].cpu().numpy(), xs[i].cpu().numpy())
        del tls, lmass, lse, h, logp
    torch.cuda.synchronize()
    assert torch.all((beta_all >= 0) & (beta_all <= 1.0 + 1e-5)).item()
    assert torch.all(torch.isfinite(e_all)).item()
    w_np = np32(w)
    ell_np = ell.cpu().numpy()
    for b, (hb, lp, xs) in check.items():
        lq = _oracle_lq(hb, w_np)
        beta_o, e_o = MX.expected_len_blocks(lq[None], ell_np[b:b + 1], wl.z_temp, xs[None],
                                             lp[None])
        assert _rel(beta_all[b].cpu().numpy(), beta_o[0]) < 1e-4
        assert _rel([e_all[b].item()], e_o) < 1e-4
        ob = OB.acceptance_objective(lq[None], ell_np[b:b + 1], wl.z_temp, xs[None], lp[None],
                                     tau=0.1)
        assert abs(nll_all[b].item() - ob["nll"][0]) < 1e-4 * max(1.0, abs(ob["nll"][0]))
        if lt_all[b].item() == ob["ell_tau"][0]:
            assert abs(j_all[b].item() - ob["J"][0]) < 1e-4 * max(1.0, abs(ob["J"][0]))
        else:   # end to end the two heads differ by ~1e-6 per log-prob: a near-tie only
            l = min(lt_all[b].item(), int(ob["ell_tau"][0]))
            assert abs(ob["log_r"][0, l - 1] - np.log(0.1)) < 1e-3
        print(f"[fullsize] objective block {b}: E={e_o[0]:.6f} ok", flush=True)
    print(f"[fullsize] objective mean E over {wl.B} blocks: {e_all.mean().item():.5f}; mean "
          f"l_tau {lt_all.float().mean().item():.2f}, mean J {j_all.mean().item():.3f}, mean NLL "
          f"{nll_all.mean().item():.3f}", flush=True)


def test_stress_workload_1000_step_loop():
    """B=256, K=8, R=4: the head, draw and verification every step for 1000 steps with a Philox
    stream per sequence; sampled (block, step) pairs checked against the oracle. The sampled
    steps also request the acceptance masses, E and AL_b, i.e. take the benchmark's verification
    stream (eight 32-tile chunks per workgroup at this shape); the others verify without them."""
    from paper_2608_05448_amd import dblast as D
    wl = synth.WORKLOADS["stress"]
    steps = 1000
    print(f"[fullsize] stress B={wl.B} K={wl.K} R={wl.R} for {steps} steps", flush=True)
    h = synth.make_h(wl, "cuda")
    w = synth.make_w(wl, "cuda")
    ell = synth.make_ell(wl, "cuda")
    logp = synth.make_logp(wl, rows=wl.K + 1, device="cuda")
    B, K = wl.B, wl.K
    probe_blocks, probe_steps = [3, 200], [0, 1, 577, 999]
    rec = {}
    z = torch.empty(B, dtype=torch.int32, device="cuda")
    x = torch.empty((B, K), dtype=torch.int32, device="cuda")
    tot_acc = torch.zeros(B, dtype=torch.float64, device="cuda")
    for t in range(steps):
        tls, lmass, lse = D.dbl_head_logprobs(h, w)
        D.dbl_sample_block(tls, lmass, lse, ell, z_temp=wl.z_temp, seed=wl.philox_seed, step=t,
                           z_out=z, x_out=x)
        full = t in probe_steps
        out = D.dbl_verify_block(tls, lmass, lse, ell, x, logp, z_temp=wl.z_temp,
                                 seed=wl.philox_seed, step=t, want_beta=full, want_al=full,
                                 want_exp_len=full)
        tot_acc += out["n_accept"].double()
        if full:
            rec[t] = (z.cpu().numpy(), x.cpu().numpy(), out["n_accept"].cpu().numpy(),
                      out["next_token"].cpu().numpy(), out["accept_mass"].cpu().numpy(),
                      out["al_expected"].cpu().numpy(), out["exp_len"].cpu().numpy())
        if t % 250 == 0:
            torch.cuda.synchronize()
            print(f"[fullsize] stress step {t}", flush=True)
    torch.cuda.synchronize()
    w_np = np32(w)
    ell_np = ell.cpu().numpy()
    lp = logp.cpu().numpy()
    for b in probe_blocks:
        o_tls, o_lm, o_ls, lq = _oracle_factored(h[b], w_np)
        for t in probe_steps:
            zo, xo = MX.sample_blocks(o_tls[None], o_lm[None], o_ls[None], ell_np[b:b + 1],
                                      wl.z_temp, wl.philox_seed, t, np.array([b]))
            zg, xg, nag, ntg, betag, alg, eg = (a[b] for a in rec[t])
            assert zg == zo[0]
            assert np.array_equal(xg, xo[0]), (b, t)
            ref = MX.verify_blocks(lq[None], ell_np[b:b + 1], wl.z_temp, xo, lp[b:b + 1],
                                   wl.philox_seed, t, np.array([b]))
            assert nag == ref["n_accept"][0] and ntg == ref["next_token"][0], (b, t)
            np.testing.assert_allclose(betag, ref["beta"][0], rtol=1e-4, atol=1e-30)
            np.testing.assert_allclose(alg, ref["al"][0], rtol=1e-4, atol=1e-30)
            np.testing.assert_allclose(eg, ref["E"][0], rtol=1e-4, atol=1e-30)
    # Different steps draw different blocks (the step counter advances every stream).
    assert not np.array_equal(rec[0][1], rec[1][1])
    print(f"[fullsize] stress mean accepted per block-step "
          f"{(tot_acc.sum() / (B * steps)).item():.4f}", flush=True)


def test_greedy_qwen3_8b_full_shape():
    """Greedy-branch step at the Qwen3-8B shape in the benchmark's configuration: the head's
    argmax on sampled rows against the oracle's binary64 argmax (certified near-ties only), then
    the greedy draw and verification for every block against the oracle fed the same branch
    tokens, at two target temperatures."""
    from oracle import greedy as GR
    from paper_2608_05448_amd import dblast as D
    wl = synth.WORKLOADS["qwen3_8b"]
    print(f"[fullsize] greedy qwen3_8b B={wl.B} K={wl.K} R={wl.R}", flush=True)
    h = synth.make_h(wl, "cuda")
    w = synth.make_w(wl, "cuda")
    ell = synth.make_ell(wl, "cuda")
    tls, lmass, lse, am = D.dbl_head_logprobs(h, w, argmax=True)
    t2, l2, s2 = D.dbl_head_logprobs(h, w)
    torch.cuda.synchronize()
    assert torch.equal(tls, t2) and torch.equal(lmass, l2) and torch.equal(lse, s2)
    xhat = am.cpu().numpy()
    w_np = np32(w)
    ties = 0
    for b in (0, 7, 15):
        logits = OH.head_logits(np32(h[b]).reshape(wl.K * wl.R, wl.d), w_np)
        want = GR.branch_tokens(logits).reshape(wl.K, wl.R)
        for k, z in zip(*np.nonzero(xhat[b] != want)):
            row = logits[k * wl.R + z]
            assert abs(row[xhat[b, k, z]] - row[want[k, z]]) <= 2e-4
            ties += 1
    print(f"[fullsize] greedy argmax certified near-ties {ties}", flush=True)
    ell_np = ell.cpu().numpy()
    seq = np.arange(wl.B)
    z, x = D.dbl_sample_greedy(am, ell, z_temp=wl.z_temp, seed=wl.philox_seed, step=3, V=wl.V)
    z_o, x_o = GR.sample_blocks_greedy(xhat, ell_np, wl.z_temp, wl.philox_seed, 3, seq)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(z.cpu().numpy(), z_o)
    np.testing.assert_array_equal(x.cpu().numpy(), x_o)
    for T in (0.0, 1.0):
        logp = synth.make_logp(wl, rows=wl.K + 1, device="cuda", temperature=T)
        out = D.dbl_verify_greedy(am, ell, x, logp, z_temp=wl.z_temp, seed=wl.philox_seed,
                                  step=3)
        torch.cuda.synchronize()
        ref = GR.verify_blocks_greedy(xhat, ell_np, wl.z_temp, x_o, logp.cpu().numpy(),
                                      wl.philox_seed, 3, seq)
        np.testing.assert_array_equal(out["n_accept"].cpu().numpy(), ref["n_accept"])
        np.testing.assert_array_equal(out["next_token"].cpu().numpy(), ref["next_token"])
        assert _rel(out["accept_mass"].cpu().numpy(), ref["beta"]) < 1e-4
        assert _rel(out["exp_len"].cpu().numpy(), ref["E"]) < 1e-4
        print(f"[fullsize] greedy T={T}: mean n_accept {out['n_accept'].float().mean().item():.3f}",
              flush=True)
