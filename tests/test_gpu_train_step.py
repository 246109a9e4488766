"""One training step through every entry point, on an adapted LM head (GPU).

forward (lora_apply: logits = base + LoRA residual) -> PPO token loss with the
action mask (lora_token_loss, bfloat16 gradient at the logits) -> lora_grad and
lora_grad_x from that gradient -> lora_adamw_step on float32 masters, writing
the table's bfloat16 weights -> forward again with the updated adapters.  Each
stage is compared with the oracle on the exact values the previous stage left
on the device, so the check is per stage (forward and gradient bar: relF <=
5e-3, max-abs <= 3e-2); it pins that the entry points' layouts compose.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_helpers import DEV, MAX_ABS, REL_FRO, effective, say
from workloads.device import case_to_device

import paper_2601_07376_amd as L

pytestmark = pytest.mark.gpu


def f32(x):
    return float(np.float32(x))


def test_train_step_composes():
    say("train step")
    case = workloads.random_case(77, 512, 256, 1024, 4, rank_choices=(8, 16, 32), layout="segments",
                                 seg_len=(16, 160), mask_p=0.5, y_dtype="f32", want_y=True)
    dev = case_to_device(case, DEV)
    table = L.Table(case.num_slots, case.d_in, case.d_out, w_dtype=torch.bfloat16, device=DEV)
    for a in range(case.num_slots):
        table.set(a, dev["A"][a], dev["B"][a], float(case.scales[a]))
    table.upload()
    plan = L.Plan(table, idx=dev["idx"], mask=dev["mask"])
    eff = effective(case)
    mask = np.asarray(case.mask)
    n, V = case.n, case.d_out
    A64 = [a.cpu().double().numpy() for a in [t.float() for t in dev["A"]]]
    B64 = [b.cpu().double().numpy() for b in [t.float() for t in dev["B"]]]
    X64 = dev["X"].float().cpu().double().numpy()

    # 1. forward: logits = base + s (X A^T) B^T
    logits = dev["Y"].clone()
    base = logits.cpu().double().numpy()
    L.apply(plan, dev["X"], logits)
    torch.cuda.synchronize()
    z = logits.cpu().double().numpy()
    ref = oracle.apply(eff, X64, base, A64, B64, case.scales)
    act = eff >= 0
    assert oracle.rel_fro(z[act] - base[act], ref[act] - base[act]) <= REL_FRO
    assert oracle.max_abs(z, ref) <= MAX_ABS

    # 2. PPO loss over the action mask, gradient at the logits in bfloat16
    rng = np.random.default_rng(78)
    target = rng.integers(0, V, n)
    _, lp, _ = oracle.token_loss(oracle.LOSS_CE, z, target, weight=np.ones(n))
    rho = rng.choice([0.6, 0.9, 1.0, 1.1, 1.4], n)
    old = (lp - np.log(rho)).astype(np.float32)
    adv = (rng.standard_normal(n) / 64).astype(np.float32)
    dz = torch.empty(n, V, dtype=torch.bfloat16, device=DEV)
    loss = torch.empty(n, device=DEV)
    tm = torch.from_numpy(mask).to(DEV)
    L.token_loss(L.LOSS_PPO, logits, torch.from_numpy(target.astype(np.int32)).to(DEV), dz, loss,
                 mask=tm, old_logp=torch.from_numpy(old).to(DEV), adv=torch.from_numpy(adv).to(DEV))
    torch.cuda.synchronize()
    rL, _, rdz = oracle.token_loss(oracle.LOSS_PPO, z, target, mask=mask, old_logp=old.astype(np.float64),
                                   adv=adv.astype(np.float64))
    assert np.allclose(loss.cpu().double().numpy(), rL, rtol=1e-4, atol=1e-6)
    dzf = dz.float().cpu().double().numpy()
    assert oracle.rel_fro(dzf, rdz) <= 4e-3             # one bfloat16 rounding per element

    # 3. gradients of the adapters and of X from the device's dlogits
    dA, dB = L.grad(plan, dev["X"], dz)
    dX = torch.zeros(n, case.d_in, device=DEV)
    L.grad_x(plan, dz, dX)
    torch.cuda.synchronize()
    rA, rB = oracle.grad(eff, mask, X64, dzf, A64, B64, case.scales)
    g = np.concatenate([t.cpu().double().numpy().ravel() for t in dA + dB])
    r = np.concatenate([x.ravel() for x in rA + rB])
    assert oracle.rel_fro(g, r) <= REL_FRO and oracle.max_abs(g, r) <= MAX_ABS
    rX = oracle.grad_x(eff, mask, dzf, A64, B64, case.scales, np.zeros((n, case.d_in)))
    gx = dX.cpu().double().numpy()
    sel = act & (mask != 0)
    assert oracle.rel_fro(gx[sel], rX[sel]) <= REL_FRO and np.all(gx[~sel] == 0)

    # 4. AdamW on float32 masters of every A_a and B_a, writing the table's weights
    params = []
    for a in range(case.num_slots):
        for w, gr in ((dev["A"][a], dA[a]), (dev["B"][a], dB[a])):
            p = w.float().reshape(-1).clone()
            params.append(dict(p=p, m=torch.zeros_like(p), v=torch.zeros_like(p),
                               g=gr.reshape(-1).contiguous(), p_bf16=w.reshape(-1), step=1,
                               lr=1e-2, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01))
    before = [(q["p"].cpu().double().numpy(), q["g"].cpu().double().numpy()) for q in params]
    L.adamw_step(params)
    torch.cuda.synchronize()
    for (p0, g0), q in zip(before, params):
        rp, _, _ = oracle.adamw(p0, 0.0, 0.0, g0, 1, f32(1e-2), f32(0.9), f32(0.999), f32(1e-8), f32(0.01))
        assert np.allclose(q["p"].cpu().double().numpy(), rp, rtol=1e-5, atol=1e-7)
        assert torch.equal(q["p_bf16"].view(torch.int16), q["p"].to(torch.bfloat16).view(torch.int16))

    # 5. forward again: the plan still names the same weight buffers, now updated
    logits2 = dev["Y"].clone()
    L.apply(plan, dev["X"], logits2)
    torch.cuda.synchronize()
    A2 = [t.float().cpu().double().numpy() for t in dev["A"]]
    B2 = [t.float().cpu().double().numpy() for t in dev["B"]]
    ref2 = oracle.apply(eff, X64, base, A2, B2, case.scales)
    z2 = logits2.cpu().double().numpy()
    assert oracle.rel_fro(z2[act] - base[act], ref2[act] - base[act]) <= REL_FRO
    assert oracle.max_abs(z2, ref2) <= MAX_ABS
    assert not np.array_equal(z2, z)                  # the step changed the adapters
