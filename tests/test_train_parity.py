"""GPU parity of the training-time DMS attention (continuous decisions,
Sec. 3.1 Eq. 1 / Fig. 1b) and of the Gumbel-sigmoid against the CPU oracle
(float64 definitions, gradients by autograd)."""
import numpy as np
import pytest

import dms_synth as sy
import oracle

pytestmark = pytest.mark.gpu

D = 128


def _bf16(x):
    return sy.f32_to_bf16_bits_np(np.asarray(x, np.float32))


def _dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _run(B, T, H, g, w, seed, alpha_kind="uniform", q_scale=1.0):
    import torch
    from paper_2506_05345_amd import dms
    rng = np.random.default_rng(seed)
    Hq = H * g
    qb = _bf16(rng.normal(0, q_scale, (B, T, Hq, D)))
    kb = _bf16(rng.normal(size=(B, T, H, D)))
    vb = _bf16(rng.normal(size=(B, T, H, D)))
    db = _bf16(rng.normal(size=(B, T, Hq, D)))
    if alpha_kind == "uniform":
        al = rng.uniform(0, 1, (B, T, H)).astype(np.float32)
        al[rng.uniform(size=al.shape) < 0.1] = 0.0
    elif alpha_kind == "near_one":
        al = np.full((B, T, H), 1.0 - 1e-6, np.float32)
    else:
        al = (rng.uniform(size=(B, T, H)) < 0.5).astype(np.float32)
    f = sy.bf16_bits_to_f32_np
    q, k, v, do = f(qb), f(kb), f(vb), f(db)
    cfg = dms.make_train_config(B, T, H, g, D, w)
    ws = torch.empty(dms.dms_train_workspace(cfg), dtype=torch.uint8, device="cuda")
    out = torch.full((B, T, Hq, D), float("nan"), device="cuda")
    lse = torch.full((B, Hq, T), float("nan"), device="cuda")
    qd, kd, vd, dd = _dev_bf16(qb), _dev_bf16(kb), _dev_bf16(vb), _dev_bf16(db)
    ad = torch.from_numpy(al).cuda()
    dms.dms_train_attention_fwd(cfg, qd, kd, vd, ad, out, lse, ws)
    dq = torch.full((B, T, Hq, D), float("nan"), device="cuda")
    dk = torch.full((B, T, H, D), float("nan"), device="cuda")
    dv = torch.full((B, T, H, D), float("nan"), device="cuda")
    da = torch.full((B, T, H), float("nan"), device="cuda")
    dms.dms_train_attention_bwd(cfg, qd, kd, vd, ad, out, lse, dd, dq, dk, dv, da, ws)
    torch.cuda.synchronize()
    O, L = oracle.train_attention(q, k, v, al.astype(np.float64), w, g)
    gq, gk, gv, ga = oracle.train_attention_grads(q, k, v, al.astype(np.float64), do, w, g)
    res = {"out": np.abs(out.cpu().numpy() - O).max(), "lse": np.abs(lse.cpu().numpy() - L).max()}
    for name, got, ref in (("dq", dq, gq), ("dk", dk, gk), ("dv", dv, gv), ("dalpha", da, ga)):
        gg = got.cpu().numpy()
        assert np.isfinite(gg).all(), name
        res[name] = np.abs(gg - ref).max() / max(1.0, np.abs(ref).max())
    return res


GRAD_TOL = 2e-2


@pytest.mark.parametrize("B,T,H,g,w,seed", [
    (1, 64, 1, 1, 16, 0), (2, 100, 2, 5, 16, 1), (1, 150, 2, 3, 40, 2), (1, 97, 1, 4, 1, 3),
    (2, 33, 1, 2, 64, 4), (1, 200, 1, 16, 7, 5), (1, 1, 1, 1, 1, 10), (3, 1, 2, 16, 4, 11),
    (1, 1024, 2, 2, 256, 12), (1, 700, 1, 8, 256, 13), (1, 257, 2, 7, 300, 14)])
def test_forward_and_backward(B, T, H, g, w, seed):
    r = _run(B, T, H, g, w, seed)
    print({k: float(f"{v:.3e}") for k, v in r.items()})
    assert r["out"] <= 1e-2 and r["lse"] <= 5e-3, r
    for name in ("dq", "dk", "dv", "dalpha"):
        assert r[name] <= GRAD_TOL, (name, r)


def test_binary_decisions_and_peaked_scores():
    r = _run(1, 120, 2, 5, 12, 7, alpha_kind="binary", q_scale=4.0)
    print(r)
    assert r["out"] <= 1e-2 and r["lse"] <= 5e-3, r
    for name in ("dq", "dk", "dv", "dalpha"):
        assert r[name] <= GRAD_TOL, (name, r)


def test_decisions_near_one_keep_gradients_finite():
    r = _run(1, 90, 1, 3, 10, 8, alpha_kind="near_one")
    print(r)
    assert r["out"] <= 1e-2
    for name in ("dq", "dk", "dv", "dalpha"):
        assert r[name] <= GRAD_TOL, (name, r)


def test_gumbel_sigmoid_forward_backward():
    import torch
    from paper_2506_05345_amd import dms
    rng = np.random.default_rng(9)
    n = 10000
    x = rng.normal(-5, 3, n).astype(np.float32)
    u = rng.uniform(1e-6, 1 - 1e-6, n).astype(np.float32)
    da = rng.normal(size=n).astype(np.float32)
    for tau in (0.05, 0.5, 1.0):
        xd, ud, dad = (torch.from_numpy(a).cuda() for a in (x, u, da))
        al = torch.empty(n, device="cuda")
        dx = torch.empty(n, device="cuda")
        dms.dms_gumbel_sigmoid_fwd(n, xd, ud, tau, al)
        dms.dms_gumbel_sigmoid_bwd(n, al, dad, tau, dx)
        torch.cuda.synchronize()
        ref = oracle.gumbel_sigmoid(x, u, tau)
        assert np.abs(al.cpu().numpy() - ref).max() < 2e-5, tau
        refd = oracle.gumbel_sigmoid_grad(al.cpu().numpy(), da, tau)
        assert np.abs(dx.cpu().numpy() - refd).max() <= 1e-5 * max(1.0, np.abs(refd).max()), tau
