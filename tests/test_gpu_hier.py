"""GPU parity of the hierarchical codec of Alg. 1 (Sec. 4.1) through the C
ABI, bit for bit against the CPU oracle on the same seeded inputs: the
anchor and correction planes, the page and chunk metadata, and the BF16
reconstruction from the anchor alone and from the merged codes.  Ragged
pages and chunks, paged pools, several alpha values, adversarial values, and
a full 32K-token Llama-3-8B layer; the biased and centred splits and the
single 4-bit code (whose encode leaves the residual planes untouched)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests.gpu_cases import bits, note, random_kv

pytestmark = pytest.mark.gpu

HMETA = ("k_gmin", "k_gscale", "k_mu", "k_sigma", "v_gmin", "v_gscale", "v_mu", "v_sigma")
VARIANTS = ("biased", "centred", "int4")


def run_case(k, v, alpha, bt=None, seed=0, variant="biased"):
    vid = oracle.H_VARIANTS[variant]
    has_res = variant != "int4"
    T, Hkv = int(k.shape[0]), int(k.shape[1])
    if bt is None:
        bt_eff, table, n_blocks = T, torch.zeros(1, 1, dtype=torch.int32), 1
    else:
        bt_eff = bt
        table, n_blocks = inputs.paged_block_table(torch.tensor([T]), bt, seed)
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt_eff, max_blocks_per_seq=table.shape[1],
                    num_blocks=n_blocks, max_tokens=T)
    OL = oracle.Layout(Hkv=Hkv, bt=bt_eff, max_blocks=table.shape[1], max_tokens=T)
    pool = lynx.KVPool.allocate(L, 1)
    hm = lynx.HMeta.empty(L, 1)
    tdev = table.cuda()
    # residual planes preset to a marker the 4-bit encode must leave alone
    pool.k_res.fill_(0x5A)
    pool.v_res.fill_(0x5A)
    note(f"hkv_encode T={T} Hkv={Hkv} alpha={alpha} bt={bt_eff} variant={variant}")
    lynx.lynx_hkv_encode(L, 0, T, tdev, k.cuda(), v.cuda(), alpha, vid, pool.k_anc, pool.v_anc,
                         pool.k_res if has_res else None, pool.v_res if has_res else None, hm)
    modes = (("anchor", False), ("full", True)) if has_res else (("anchor", False),)
    if has_res:
        pool.merge()
    outs = {}
    for mode, full in modes:
        ko = torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device="cuda")
        vo = torch.empty_like(ko)
        kp, vp = (pool.k_codes, pool.v_codes) if full else (pool.k_anc, pool.v_anc)
        note(f"hkv_dequant {mode} T={T} variant={variant}")
        lynx.lynx_hkv_dequant(L, 0, T, tdev, full, kp, vp, alpha, vid, hm, ko, vo)
        outs[mode] = (bits(ko), bits(vo))
    torch.cuda.synchronize()
    # the oracle on the same inputs
    nbytes = oracle.plane_bytes(OL, n_blocks, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    planes["k_res"][:] = 0x5A   # as preset on the device: rows no token maps to keep it
    planes["v_res"][:] = 0x5A
    ohm = oracle.HMeta.empty(OL, 1)
    oracle.hencode(OL, 0, T, table.numpy(), bits(k), bits(v), alpha, planes, ohm, variant)
    for name in ("k_anc", "v_anc", "k_res", "v_res"):
        got = getattr(pool, name).cpu().numpy()
        assert np.array_equal(got, planes[name]), f"{name}: {np.count_nonzero(got != planes[name])} bytes differ"
    for name in HMETA:
        got = getattr(hm, name).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), getattr(ohm, name).view(np.uint32)), name
    ref = {"anchor": oracle.hdequant("anchor", OL, 0, T, table.numpy(), planes["k_anc"], planes["v_anc"],
                                     alpha, ohm, variant)}
    if has_res:
        codes = {p: oracle.merge(planes[p + "_anc"], planes[p + "_res"]) for p in ("k", "v")}
        ref["full"] = oracle.hdequant("full", OL, 0, T, table.numpy(), codes["k"], codes["v"], alpha, ohm,
                                      variant)
    for mode, _ in modes:
        for i, name in enumerate(("K", "V")):
            got, want = outs[mode][i], ref[mode][i]
            assert np.array_equal(got, want), f"{mode} {name}: {np.count_nonzero(got != want)} values differ"


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("T,Hkv,alpha", [(1, 1, 255.0), (31, 2, 1.0), (32, 1, 15.0), (256, 2, 255.0),
                                         (257, 1, 15.0), (1000, 4, 255.0), (600, 2, 1e-6)])
def test_hier_contiguous(T, Hkv, alpha, variant):
    k, v = random_kv(T, Hkv, seed=2000 + T)
    run_case(k, v, alpha, variant=variant)


@pytest.mark.parametrize("alpha", [1e-4, 9.99e-4, 1e-3, 0.01, 0.3, 3.0, 1e4, 1e30])
def test_hier_alpha_range(alpha):
    """The encode finds each code from the transform's fp32 value and one
    exact step against the thresholds around it; across the range of alpha
    (both sides of the switch to the linear first guess at 1e-3) the codes
    stay those the oracle's thresholds decide."""
    k, v = random_kv(2048, 2, seed=2200)
    run_case(k, v, alpha, variant="centred")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("T,bt", [(700, 16), (513, 32), (129, 8)])
def test_hier_paged(T, bt, variant):
    k, v = random_kv(T, 2, seed=2100 + T)
    run_case(k, v, 255.0, bt=bt, seed=T, variant=variant)


def test_hier_adversarial():
    """Constant and two-valued channels, signed zeros, denormals, huge values,
    a constant chunk inside a varying page, and exact sign-of-zero cases."""
    T, Hkv = 300, 2
    g = torch.Generator().manual_seed(11)
    x = torch.randn(T, Hkv, 128, generator=g)
    x[:, 0, 0] = 3.25
    x[:, 0, 1] = torch.where(torch.arange(T) % 3 == 0, -7.0, 9.0)
    x[:, 0, 2] = -0.0
    x[:, 0, 3] = torch.randn(T, generator=g) * 1e-39
    x[:, 1, 4] = torch.randn(T, generator=g) * 1e37
    x[32:64, 1, 5] = 0.75                 # one constant chunk
    x[:, 1, 6] = torch.arange(T) % 5      # small integers: exact means and ties
    v = torch.randn(T, Hkv, 128, generator=g)
    v[:, :, 7] = 1.5
    for variant in VARIANTS:
        run_case(x.to(torch.bfloat16), v.to(torch.bfloat16), 255.0, variant=variant)
        run_case(x.to(torch.bfloat16), v.to(torch.bfloat16), 1.0, variant=variant)


@pytest.mark.parametrize("variant", VARIANTS)
def test_hier_llama3_8b_layer(variant):
    w = inputs.WORKLOADS["llama3-8b-32k"]
    k = inputs.kv(w, "k", layer=5)
    v = inputs.kv(w, "v", layer=5)
    run_case(k, v, 255.0, variant=variant)
