"""Dense controls of the decode benchmark (the dense control of Sec. 6.3's
canary) on the GPU:

* all-FP8 control: the same KV with no Retier, every page FP8, attended by the
  mixed-format decode kernel; compared with the oracle within 1e-3;
* all-bf16 control: the KV as bf16 pages attended by the control kernel;
  compared within 1e-3 with dense softmax attention written out in numpy
  (fp64) over the same bf16 keys and values.
"""
import dataclasses

import numpy as np
import pytest

import mkv_workloads as wl
from _harness import max_abs

pytestmark = pytest.mark.gpu

TOL = 1e-3
PAGE = 16


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available()
    import paper_2608_23834_amd as mk
    mk.lib()
    return torch


def test_all_fp8_control_long_pair(torch_cuda):
    """The long pair at full size (2 x 59,008 tokens, one layer) with every
    page left FP8 (no Retier): decode against the oracle."""
    from _harness import Twin
    w = wl.workload(3)
    tw = Twin(w, lens=list(w.ctx))
    tw.fill()
    tw.check_tables()
    assert (tw.otags == 0).all()
    res = tw.decode()
    err = max(max_abs(res["out"], res["ref_out"]), max_abs(res["lse"], res["ref_lse"]))
    print(f"\n  all-FP8 long pair: max|dO|, max|dlse| {err:.3e}", flush=True)
    assert np.all(np.isfinite(res["out"])) and err <= TOL


def _dense_ref(q, k, v, lens, G):
    """softmax(q k^T / sqrt(d)) v per request and query head, fp64, from bf16."""
    qf = wl.bf16_to_f32(q).astype(np.float64)
    kf = wl.bf16_to_f32(k).astype(np.float64)
    vf = wl.bf16_to_f32(v).astype(np.float64)
    d = q.shape[-1]
    out = np.zeros(q.shape)
    lse = np.zeros(q.shape[:2])
    cu = np.r_[0, np.cumsum(lens)]
    for r, L in enumerate(lens):
        for hq in range(q.shape[1]):
            s = kf[cu[r]:cu[r] + L, hq // G] @ qf[r, hq] / np.sqrt(d)
            m = s.max()
            e = np.exp(s - m)
            out[r, hq] = e @ vf[cu[r]:cu[r] + L, hq // G] / e.sum()
            lse[r, hq] = m + np.log(e.sum())
    return out, lse


def _control_case(torch, w, lens, seed):
    import paper_2608_23834_amd as mk
    n_req, H, G, d = len(lens), w.n_kv_heads, w.n_q_heads // w.n_kv_heads, w.head_dim
    mp = max((L + PAGE - 1) // PAGE for L in lens)
    n_pages = sum((L + PAGE - 1) // PAGE for L in lens) + 3
    rng = np.random.default_rng(seed)
    ids = rng.permutation(n_pages)
    bt = np.full((n_req, mp), -1, np.int32)
    k0 = 0
    for r, L in enumerate(lens):
        npg = (L + PAGE - 1) // PAGE
        bt[r, :npg] = ids[k0:k0 + npg]
        k0 += npg
    ks, vs = zip(*(wl.kv_layer(w, 0, L, token_offset=r * 1_000_000) for r, L in enumerate(lens)))
    k, v = np.concatenate(ks), np.concatenate(vs)
    q = wl.q_decode(w, 0)
    q = np.ascontiguousarray(np.resize(q, (n_req,) + q.shape[1:]))
    ctl = mk.ControlBf16(1, w.n_q_heads, H, d, n_pages)
    btg = torch.from_numpy(bt).cuda()
    cu = torch.tensor(np.r_[0, np.cumsum(lens)], dtype=torch.int32, device="cuda")
    ctl.write(0, btg, torch.zeros(n_req, dtype=torch.int32, device="cuda"), cu,
              torch.from_numpy(k.view(np.int16)).cuda(), torch.from_numpy(v.view(np.int16)).cuda())
    out = torch.full((n_req, w.n_q_heads, d), float("nan"), device="cuda")
    lse = torch.full((n_req, w.n_q_heads), float("nan"), device="cuda")
    ws = ctl.workspace(n_req, mp)
    ws.view(torch.uint8).fill_(0xFF)  # NaN bits: the call must not depend on them
    ctl.decode(0, torch.from_numpy(q.view(np.int16)).cuda(), btg,
               torch.tensor(lens, dtype=torch.int32, device="cuda"), out, lse, ws)
    torch.cuda.synchronize()
    ref_o, ref_l = _dense_ref(q, k, v, lens, G)
    err = max(max_abs(out.cpu().numpy(), ref_o), max_abs(lse.cpu().numpy(), ref_l))
    print(f"\n  bf16 control {w.name} lens={lens[:4]}: max|dO|, max|dlse| {err:.3e}", flush=True)
    assert np.all(np.isfinite(out.cpu().numpy())) and err <= TOL


def test_bf16_control_ragged(torch_cuda):
    """Ragged lengths (1, 17, 700, 3000, partial pages), d = 256 with six and
    with twelve query heads per KV head, d = 128 with eight."""
    torch = torch_cuda
    _control_case(torch, wl.workload(2), [1, 17, 700, 3000], 1)
    _control_case(torch, dataclasses.replace(wl.workload(2), n_kv_heads=2, name="group12"),
                  [33, 2000, 5], 2)
    _control_case(torch, wl.workload(1), [2048, 100], 3)


def test_bf16_control_long_pair(torch_cuda):
    """The long pair at full size (2 x 59,008 tokens), one layer."""
    w = wl.workload(3)
    _control_case(torch_cuda, w, list(w.ctx), 4)
