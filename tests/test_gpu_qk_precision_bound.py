"""A bound on decode attention derived from the QK^T instruction's own error,
held on the one case that missed the 2e-3 absolute bar in a 1 040-seed
random sweep: a cascade case (6 sequences, 16 query heads on 1 kv head,
contexts 506, 0, 191, 192, 434, 265, a 192-token shared prefix, BF16 query,
partition 256, seed 106039).  With V unrotated (Algorithm 1 as printed) its
worst element is off by 2.5e-3 on an output of -14.09, with V rotated by
3.0e-3; relative L2 stays near 2e-5.

The cause is the QK^T instruction, not the kernel's softmax or PV: the scaled
FP4 x FP8 matrix instruction does not always return the exactly rounded dot
product; its error stays below 2^-10.5 of the largest product of the dot
product on any operands measured, and below 2^-12.5 on operands like the
kernel's (tests/test_gpu_instruction_precision.py).  In this row it returned
two of the top scores (140.98 and 140.82, nearly equal, over tokens whose V
differ by 60) 2^-9 low, 2^-14.6 of the largest product.  A score error ds_j
moves the softmax weight p_j by sigma ds_j p_j (sigma = softmax scale), so to
first order the output moves by

    delta = sigma sum_j p_j ds_j (u_j - o),
    |delta_c| <= B_c = sigma sum_j p_j eta_j |u_jc - o_c|,
    eta_j = 2^-10.5 max_d |q8_d k_jd|,

with u_j token j's V in the output basis (R v_j when V is stored rotated,
since the output is rotated back by the orthonormal R).  The bound is large
where two near-equal top scores carry very different V.  The test holds the
case, plain and cascade, in both modes, to max-abs 2e-3 + 2 B_c per element
(twice the first-order term: second-order terms and the two-term P split,
which alone gives 4.8e-5 here) and to the relative-L2 bar 1e-3.  The kernel
is deterministic, so each variant's own error is also held to a guard 20 %
above it, to catch a regression the looser derived bound would let
through."""
import math

import numpy as np
import pytest
import torch
from scipy.linalg import hadamard

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3
ETA = 2.0 ** -10.5        # instruction error bound per largest product (measured, see the module docstring)
GUARD = {False: 3e-3, True: 3.6e-3}   # the case's own max-abs error: 2.5e-3 unrotated, 3.0e-3 rotated
CASE = dict(batch=6, hq=16, hkv=1, ctx=[506, 0, 191, 192, 434, 265], prefix=192, part=256, seed=106039)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def build(uq, rotate_v, dev):
    c = CASE
    wl = workloads.custom(c["batch"], c["hq"], c["hkv"], c["ctx"], seed=c["seed"], paging="random",
                          shared_prefix_tokens=c["prefix"], rotate_v=rotate_v)
    desc = uq.CacheDesc(num_kv_heads=c["hkv"], num_pages=wl.num_pages, rotate_v=rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0x5A)
    pools = oracle.alloc_pools(wl.num_pages, c["hkv"], fill=0x5A)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        sl = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(sl, device=dev), codes, scales)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), sl, wl.num_pages, rotate_v=rotate_v, pools=pools)
    torch.cuda.synchronize()
    return wl, desc, codes, scales, pools


def first_order_bound(wl, pools, q, scale, rotate_v):
    """B[b, h, c] = sigma sum_j p_j eta_j |u_jc - o_c| over the oracle's own
    dequantised cache and query bytes, u_j = R v_j with rotate_v (R =
    H_128 / sqrt(128), symmetric), else v_j."""
    R = hadamard(128) / math.sqrt(128)
    B = np.zeros((wl.batch, wl.num_q_heads, 128))
    G = wl.num_q_heads // wl.num_kv_heads
    for b in range(wl.batch):
        n = int(wl.context_lens[b])
        if n == 0:
            continue
        for hk in range(wl.num_kv_heads):
            K = np.stack([oracle.dequant_vector(pools, wl.num_kv_heads, int(wl.page_table[b, j // 16]), hk, 0, j % 16)
                          for j in range(n)])
            V = np.stack([oracle.dequant_vector(pools, wl.num_kv_heads, int(wl.page_table[b, j // 16]), hk, 1, j % 16)
                          for j in range(n)])
            U = V @ R if rotate_v else V
            for g in range(G):
                h = hk * G + g
                q8 = np.array([oracle.e4m3_value(x) for x in oracle.prepare_query(q[b, h].reshape(1, 128))[0]])
                s = K @ q8 * scale
                p = np.exp(s - s.max())
                p /= p.sum()
                o = p @ U
                eta = ETA * np.abs(K * q8[None, :]).max(axis=1)
                B[b, h] = scale * (p * eta) @ np.abs(U - o[None, :])
    return B


@pytest.mark.parametrize("rotate_v", [False, True])
@pytest.mark.parametrize("cascade", [False, True])
def test_within_bound_derived_from_qk_instruction(uq, cascade, rotate_v):
    dev = torch.device("cuda:0")
    wl, desc, codes, scales, pools = build(uq, rotate_v, dev)
    c = CASE
    log(f"QK precision case (seed {c['seed']}): rotate_v={rotate_v}, {'cascade' if cascade else 'plain'} decode")
    q = wl.q.to(torch.bfloat16)
    scale = 1 / math.sqrt(128)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    if cascade:
        pre = uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                              torch.as_tensor(wl.prefix_lens(), device=dev), wl.shared_prefix_tokens)
        out = uq.decode_cascade(desc, q.to(dev), codes, scales, pt, ctx, wl.max_context, pre, scale, c["part"])
    else:
        out = uq.decode_attention(desc, q.to(dev), codes, scales, pt, ctx, wl.max_context, scale, c["part"])
    torch.cuda.synchronize()
    out = out.cpu().numpy().astype(np.float64)
    qf = q.float().numpy()
    ref = oracle.decode_attention(qf, pools, wl.page_table, wl.context_lens, 1, scale, rotate_v)
    bound = first_order_bound(wl, pools, qf, scale, rotate_v)
    err = np.abs(out - ref)
    rel = np.linalg.norm(out - ref) / np.linalg.norm(ref)
    worst = np.unravel_index(np.argmax(err), err.shape)
    log(f"  max-abs {err.max():.3e} at {worst} (output {ref[worst]:.4f}, first-order bound there "
        f"{bound[worst]:.3e}), rel-L2 {rel:.3e}, largest |output| {np.abs(ref).max():.1f}")
    assert np.all(np.isfinite(out))
    assert np.all(err <= MAX_ABS + 2 * bound), float((err - MAX_ABS - 2 * bound).max())
    assert err.max() <= GUARD[rotate_v]
    assert rel <= REL_L2
    assert np.all(out[1] == 0)   # the empty context
