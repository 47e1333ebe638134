"""Every federation group ends a round holding the same shard, bit for bit
(Section 4.2; Section 2, Federated Learning).  G groups start the round from
one global model, each with its own optimiser state and its own gradients.
They run their local steps, exchange their bf16 working copies and average.
Each group's fl_round, with itself as the own replica, must then give the
same master and working copy as every other group's; m and v stay local.
These are properties, so no oracle value is involved."""
import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

HP = dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


def _say(*a):
    print("[gpu-groups]", *a, flush=True)


@pytest.fixture(scope="module")
def env():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_20359_amd as P

    P.lib()
    return dict(torch=torch, P=P)


def _fill(torch, n, kind, stream, std, seed=9):
    bf16 = kind in (synth.NORMAL_BF16, synth.DRIFT_BF16, synth.STUDENT3_BF16)
    t = torch.empty(n, dtype=torch.bfloat16 if bf16 else torch.float32, device="cuda")
    synth.dev_fill(t, synth.spec(kind, stream, seed, 0.0, std))
    return t


def _eq(a, b):
    import torch

    return torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("n,G,R,A", [(300_007, 5, 4, 3), (4099, 3, 8, 1), (1, 2, 1, 2)])
def test_groups_end_bit_identical(env, n, G, R, A):
    torch, P = env["torch"], env["P"]
    _say("n=%d G=%d R=%d A=%d" % (n, G, R, A))
    r = np.random.default_rng(n + G)
    k = int(min(n, 20))
    cuts = np.sort(r.choice(np.arange(1, n), size=k - 1, replace=False)) if k > 1 else []
    off = np.concatenate([[0], cuts, [n]]).astype(np.int64)
    flags = r.integers(0, 2, off.size - 1).astype(np.uint8)
    lay = P.Layout(off, flags)
    weights = r.uniform(0.5, 4.0, G).astype(np.float32)
    step0 = int(r.integers(1, 50))

    # the global model every group starts the round from
    master0 = _fill(torch, n, synth.NORMAL_F32, 1, 0.02)
    working0 = master0.to(torch.bfloat16)
    grads, m0, v0 = [], [], []
    for g in range(G):
        grads.append([_fill(torch, n, synth.NORMAL_BF16, 1000 + 64 * g + j, 1e-3)
                      for j in range(A * R)])
        m0.append(_fill(torch, n, synth.NORMAL_F32, 200 + g, 1e-4))
        v0.append(_fill(torch, n, synth.NORMAL_F32, 300 + g, 1e-3) ** 2)

    # each group's local steps, giving the working copies the groups exchange
    sent = []
    for g in range(G):
        master, working = master0.clone(), working0.clone()
        m, v = m0[g].clone(), v0[g].clone()
        for a in range(A):
            P.fl_local_step(lay, HP, step0 + a, grads[g][a * R:(a + 1) * R], 1.0 / R, master, m,
                            v, working)
        sent.append(working)

    # each group's whole round, with its own working copy as the own replica
    out = []
    for g in range(G):
        master, working = master0.clone(), working0.clone()
        m, v = m0[g].clone(), v0[g].clone()
        cfg = P.make_round_cfg(R, G, A, weights, HP, self_group=g, grad_scale=1.0 / R,
                               step0=step0)
        reps = [None if j == g else sent[j] for j in range(G)]
        P.fl_round(lay, cfg, grads[g], reps, master, m, v, working)
        out.append((master, m, v, working))

    # the average of the exchanged copies, as one standalone FedAvg
    fa_master = torch.empty_like(master0)
    fa_working = torch.empty_like(working0)
    P.fl_fedavg(lay, sent, weights, fa_master, fa_working)
    torch.cuda.synchronize()

    for g in range(G):
        assert _eq(out[g][0], fa_master), "group %d master differs from the FedAvg" % g
        assert _eq(out[g][3], fa_working), "group %d working copy differs" % g
    assert _eq(fa_working, fa_master.to(torch.bfloat16))
    if n > 1:
        for g in range(1, G):
            assert not _eq(out[g][1], out[0][1]), "m is not group-local"
            assert not _eq(out[g][2], out[0][2]), "v is not group-local"
    lay.close()
