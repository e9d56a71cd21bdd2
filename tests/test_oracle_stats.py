"""Pins of the oracle's producers of the selection signals (Sec. 5.3 u, d_in, d_out; Sec. 3
confidence) against torch's library softmax / log-softmax on the CPU in fp64."""
import numpy as np
import torch

import oracle


def test_token_stats_against_log_softmax():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((37, 501)) * 3
    x[5, 17] = x[5, 300] = x[5].max() + 1.0  # tied maximum: the smaller index wins
    y = rng.integers(0, 501, 37).astype(np.int32)
    logp, conf, amax = oracle.token_stats(x, y)
    ls = torch.log_softmax(torch.from_numpy(x), dim=-1)
    np.testing.assert_allclose(logp, ls[np.arange(37), y].numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(conf, ls.exp().max(dim=-1).values.numpy(), rtol=1e-13)
    assert amax[5] == 17
    assert (amax == np.argmax(x, axis=-1)).all()


def test_attn_stats_against_library_softmax_on_views():
    rng = np.random.default_rng(1)
    B, Hq, Hkv, L, d, r0 = 2, 4, 2, 20, 8, 8
    Lr = L - r0
    q = rng.standard_normal((B, Hq, L, d))
    kl, kc = rng.standard_normal((B, Hkv, L, d)), rng.standard_normal((B, Hkv, L, d))
    si = np.array([[9, 12, 15], [8, 19, -1]], np.int32)
    ns = np.array([3, 2], np.int32)
    masked = rng.integers(0, 2, (B, Lr)).astype(np.uint8)
    drafted = (rng.integers(0, 3, (B, Lr)) == 0).astype(np.uint8)
    d_in, d_out = oracle.attn_stats(q, kl, kc, si, ns, r0, masked, drafted)
    for b in range(B):
        S = set(si[b, : ns[b]].tolist())
        A = torch.zeros(L, L, dtype=torch.float64)
        for h in range(Hq):
            g = h // 2
            for i in range(L):
                K = torch.from_numpy(kl[b, g]).clone()
                for j in S:
                    if j != i:
                        K[j] = torch.from_numpy(kc[b, g, j])  # override off the diagonal
                A[i] += torch.softmax(K @ torch.from_numpy(q[b, h, i]) / np.sqrt(d), 0) / Hq
        Ar = A[r0:, r0:].numpy()
        np.testing.assert_allclose(d_in[b], (Ar * masked[b][:, None]).sum(0), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(d_out[b], (Ar * drafted[b][None, :]).sum(1), rtol=1e-12, atol=1e-14)
