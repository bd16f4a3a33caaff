"""arckv_attend_noalloc against arckv_attend: the same kernels on the same
partition, with the partials in the library's static per-GPU scratch instead of
a workspace, so the outputs must be equal bit for bit.  Two calls in a row, the
second smaller, so the second reuses the array the first left behind; plus the
float64 definition (eq. concatenated_attention_preservation) on sampled pairs."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


def A():
    from paper_2609_36835_amd import arckv
    return arckv


def _inputs(P, G, t, F, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    bf = dict(device="cuda", dtype=torch.bfloat16)
    Q = torch.randn(P, G, 128, generator=g, **bf)
    Ck = torch.randn(P, t, 128, generator=g, **bf) if t else None
    Cv = torch.randn(P, t, 128, generator=g, **bf) if t else None
    beta = (torch.rand(P, t, device="cuda", generator=g) * 6 - 3) if t else None
    Kf = torch.randn(P, F, 128, generator=g, **bf) if F else None
    Vf = torch.randn(P, F, 128, generator=g, **bf) if F else None
    return Q, Ck, beta, Cv, Kf, Vf


def _np(x):
    return None if x is None else x.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("shapes", [[(512, 4, 6554, 300), (64, 2, 1000, 0)], [(128, 8, 0, 4097), (3, 1, 5, 2)]])
def test_attend_noalloc_matches_attend(shapes):
    for i, (P, G, t, F) in enumerate(shapes):
        print(f"  call {i}: P={P} G={G} t={t} F={F}", flush=True)
        Q, Ck, beta, Cv, Kf, Vf = _inputs(P, G, t, F, seed=17 + i)
        ref = A().attend(Q, Ck, beta, Cv, Kf, Vf)
        out = A().attend_noalloc(Q, Ck, beta, Cv, Kf, Vf)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), (P, G, t, F, (out - ref).abs().max().item())
        for p in (0, P - 1):
            o64 = oracle.attend_joint(_np(Q[p]), _np(Ck[p]) if t else None, _np(beta[p]) if t else None,
                                      _np(Cv[p]) if t else None, _np(Kf[p]) if F else None,
                                      _np(Vf[p]) if F else None, 128 ** -0.5)
            err = oracle.row_rel_err(_np(out[p]), o64).max()
            assert err <= 1e-5, (p, err)


def test_attend_noalloc_rejects_beyond_scratch():
    Q, Ck, beta, Cv, _, _ = _inputs(512, 4, 16129, 0, seed=3)
    with pytest.raises(A().ArckvError) as e:
        A().attend_noalloc(Q, Ck, beta, Cv)
    assert e.value.status == A().ERR_WORKSPACE
    # a call that fits still works afterwards
    Q, Ck, beta, Cv, _, _ = _inputs(8, 4, 700, 0, seed=4)
    assert torch.equal(A().attend_noalloc(Q, Ck, beta, Cv), A().attend(Q, Ck, beta, Cv))
