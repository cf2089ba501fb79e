"""moe_permute_noalloc (the library's own scratch, no workspace argument) against
moe_permute (the caller's workspace), through the C ABI on the GPU.

Calls in a row on one GPU share the scratch, which keeps the previous call's
contents: a long batch first, then shorter ones (the second still on the
multi-launch path that uses the scratch, the third on the one-workgroup path),
so a kernel that read stale block counts would show.  Every output must equal
moe_permute's bit for bit, and the row maps the oracle's.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_08782_amd import moe, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    moe.load_library()
    yield


def _routing(T, E, k, seed):
    rng = np.random.default_rng(seed)
    L = (rng.standard_normal((T, E)) + np.linspace(1.5, 0.0, E)[None, :]).astype(np.float32)
    idx, gate = moe.moe_route_topk(None, None, None, k, logits=torch.from_numpy(L).cuda(),
                                   logits_in=True)[1:]
    counts = moe.moe_expert_histogram(idx, E)[0]
    return idx, gate, counts


def test_noalloc_permute_equals_the_workspace_permute_on_calls_in_a_row():
    E, k, G, dev = 48, 4, 3, 1
    cfg = synth.custom_config(d=128, E=E, k=k, f=64, G=G, replicas=2, zipf=1.2)
    pi = synth.popularity_perm(cfg, 0)
    pl = synth.placement_map(cfg, pi)
    for T in (5000, 1500, 300):
        print("[noalloc] T=%d" % T, flush=True)
        X = synth.normal((T, cfg.d), 7, "X", T, 1.0, "cuda", torch.bfloat16)
        idx, gate, counts = _routing(T, E, k, T)
        ref = moe.moe_permute(X, idx, gate, counts, pl, dev, E=E)
        got = moe.moe_permute(X, idx, gate, counts, pl, dev, E=E, noalloc=True)
        torch.cuda.synchronize()
        N = int(ref["group_offsets"][-1])
        for key in ("group_offsets", "token_row", "send_counts"):
            assert torch.equal(got[key], ref[key]), key
        for key in ("row_token", "row_gate", "x_perm"):
            assert torch.equal(got[key][:N], ref[key][:N]), key
        pm = oracle.permute(X.float().cpu().numpy(), idx.cpu().numpy(),
                            gate.double().cpu().numpy(), E, pl, dev)
        np.testing.assert_array_equal(got["group_offsets"].cpu().numpy(), pm["group_offsets"])
        np.testing.assert_array_equal(got["row_token"][:N].cpu().numpy(), pm["row_token"])
        np.testing.assert_array_equal(got["token_row"].cpu().numpy(), pm["token_row"])
