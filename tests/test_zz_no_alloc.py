"""attr_project_noalloc (the projection with the library's static per-GPU
scratch instead of a caller workspace) against attr_project on the same
inputs: two calls in a row, the second with a smaller input, each equal bit
for bit to attr_project (same kernels, deterministic) and within the bf16
bar of the fp64 oracle; a call too large for the scratch is rejected."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
import synth
from tests._util import dev, host, row_rel_l2, say

pytestmark = pytest.mark.gpu


def _case(seed, n, T, shapes, k):
    """Packed ragged token rows of bf16 modules (q/k/v-like sharing of one
    input among the first two modules), lengths in [0, T]."""
    rng = np.random.default_rng(seed)
    lengths = rng.integers(0, T + 1, n)
    lengths[0], lengths[-1] = T, 0
    offs = np.concatenate([[0], np.cumsum(lengths)[:-1]]).astype(np.int64)
    rows = int(lengths.sum()) + 1
    host_mods, mods = [], []
    shared = None
    for m, (d_in, d_out) in enumerate(shapes):
        a = synth.to_bf16_bits(rng.standard_normal((rows, d_in)))
        if m == 1 and shapes[0][0] == d_in:
            a = host_mods[0][0]
        g = synth.to_bf16_bits(rng.standard_normal((rows, d_out)) * 1e-2)
        R = synth.to_bf16_bits(rng.standard_normal((d_out, k)) / np.sqrt(k))
        S = synth.to_bf16_bits(rng.standard_normal((d_in, k)) / np.sqrt(k))
        host_mods.append((a, g, R, S))
        ad = shared if (m == 1 and shared is not None and shapes[0][0] == d_in) else dev(a)
        if m == 0:
            shared = ad
        mods.append(P.Module(ad, dev(g), dev(R), dev(S), out_col=m * k * k))
    return host_mods, mods, lengths, offs


def _oracle(host_mods, k, n, T, lengths, offs):
    blocks = []
    for (a, g, R, S) in host_mods:
        pad = lambda x: np.concatenate([x, np.zeros((T, x.shape[1]), x.dtype)])
        ap, gp = pad(a), pad(g)
        a3 = np.stack([ap[offs[i]:offs[i] + T] for i in range(n)])
        g3 = np.stack([gp[offs[i]:offs[i] + T] for i in range(n)])
        blocks.append(O.project(a3, g3, R, S, length=lengths))
    return O.project_concat(blocks)


def test_noalloc_matches_workspace_call_twice_then_smaller():
    k = 16
    cases = [(91, 24, 700, [(256, 512), (256, 768), (512, 256)]),     # larger first
             (92, 5, 300, [(128, 128), (192, 64)])]                  # then smaller
    for seed, n, T, shapes in cases:
        say(f"case: noalloc seed={seed} n={n} T={T} modules={len(shapes)}")
        host_mods, mods, lengths, offs = _case(seed, n, T, shapes, k)
        D = len(shapes) * k * k
        L = torch.from_numpy(lengths.astype(np.int32)).cuda()
        ro = torch.from_numpy(offs).cuda()
        ref = torch.full((n, D + 16), -3.0, dtype=torch.float32, device="cuda")
        got = torch.full((n, D + 16), 5.0, dtype=torch.float32, device="cuda")
        P.attr_project(mods, k, n, T, ref, row_offset=ro, length=L)
        P.attr_project_noalloc(mods, k, n, T, got, row_offset=ro, length=L)
        torch.cuda.synchronize()
        r, g_ = host(ref), host(got)
        np.testing.assert_array_equal(g_[:, :D], r[:, :D])
        assert (g_[:, D:] == 5.0).all(), "columns outside the module blocks were written"
        err = row_rel_l2(g_[:, :D], _oracle(host_mods, k, n, T, lengths, offs))
        say("max row rel-L2 vs oracle", err.max())
        assert err.max() <= 2e-2


def test_noalloc_rejects_calls_beyond_the_scratch():
    say("case: noalloc oversize call")
    k, n, T = 64, 5000, 64
    a = torch.zeros((n * T, 64), dtype=torch.bfloat16, device="cuda")
    R = torch.zeros((64, k), dtype=torch.bfloat16, device="cuda")
    out = torch.full((n, k * k), 1.0, dtype=torch.float32, device="cuda")
    with pytest.raises(P.AttrError) as ei:
        P.attr_project_noalloc([P.Module(a, a, R, R, 0)], k, n, T, out)
    assert ei.value.status == 4
    torch.cuda.synchronize()
    assert (out == 1.0).all().item()
