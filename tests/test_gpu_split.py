"""GPU parity of the split widths other than 4 + 4 (A-bit anchors, (8 - A)-bit
residuals, A in 2, 4, 6) through the C ABI, bit for bit against the CPU
oracle on the same seeded inputs: the anchor and residual planes, the
metadata, the merged codes (which must equal the 4 + 4 codes), and the BF16
anchor pages; contiguous and paged pools, ragged lengths, a 32K-token
Llama-3-8B layer, and verification over codes merged from 2 + 6 planes."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests.gpu_cases import bits, note, random_kv

pytestmark = pytest.mark.gpu


def run_case(k, v, A, bt=None, seed=0):
    T, Hkv = int(k.shape[0]), int(k.shape[1])
    R = 8 - A
    if bt is None:
        bt_eff, table, n_blocks = T, torch.zeros(1, 1, dtype=torch.int32), 1
    else:
        bt_eff = bt
        table, n_blocks = inputs.paged_block_table(torch.tensor([T]), bt, seed)
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt_eff, max_blocks_per_seq=table.shape[1],
                    num_blocks=n_blocks, max_tokens=T)
    OL = oracle.Layout(Hkv=Hkv, bt=bt_eff, max_blocks=table.shape[1], max_tokens=T)
    n_rows = n_blocks * Hkv * bt_eff
    dev = "cuda"
    planes = {"k_anc": torch.zeros(n_rows * 16 * A, dtype=torch.uint8, device=dev),
              "v_anc": torch.zeros(n_rows * 16 * A, dtype=torch.uint8, device=dev),
              "k_res": torch.zeros(n_rows * 16 * R, dtype=torch.uint8, device=dev),
              "v_res": torch.zeros(n_rows * 16 * R, dtype=torch.uint8, device=dev)}
    meta = lynx.Meta.empty(L, 1)
    tdev = table.cuda()
    note(f"kv_encode_split A={A} T={T} Hkv={Hkv} bt={bt_eff}")
    lynx.lynx_kv_encode_split(L, A, 0, T, tdev, k.cuda(), v.cuda(), planes["k_anc"], planes["v_anc"],
                              planes["k_res"], planes["v_res"], meta)
    codes = {w: torch.empty(n_rows * 128, dtype=torch.uint8, device=dev) for w in ("k", "v")}
    note(f"kv_merge_split A={A} rows={n_rows}")
    for w in ("k", "v"):
        lynx.lynx_kv_merge_split(A, planes[w + "_anc"], planes[w + "_res"], codes[w])
    ko = torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device=dev)
    vo = torch.empty_like(ko)
    note(f"kv_dequant_anchor_split A={A} T={T}")
    lynx.lynx_kv_dequant_anchor_split(L, A, 0, T, tdev, planes["k_anc"], planes["v_anc"], meta, ko, vo)
    torch.cuda.synchronize()
    # the oracle on the same inputs
    op = {name: np.zeros(t.numel(), np.uint8) for name, t in planes.items()}
    om = oracle.Meta.empty(OL, 1)
    oracle.encode_split(A, OL, 0, T, table.numpy(), bits(k), bits(v), op, om)
    for name in op:
        got = planes[name].cpu().numpy()
        assert np.array_equal(got, op[name]), f"{name}: {np.count_nonzero(got != op[name])} bytes differ"
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        assert np.array_equal(getattr(meta, name).cpu().numpy().view(np.uint32),
                              getattr(om, name).view(np.uint32)), name
    for w in ("k", "v"):
        want = oracle.merge_split(A, op[w + "_anc"], op[w + "_res"])
        assert np.array_equal(codes[w].cpu().numpy(), want), f"{w} codes"
    rk, rv = oracle.dequant_anchor_split(A, OL, 0, T, table.numpy(), op["k_anc"], op["v_anc"], om)
    assert np.array_equal(bits(ko), rk) and np.array_equal(bits(vo), rv)
    return codes, meta, L, tdev


@pytest.mark.parametrize("A", [2, 4, 6])
@pytest.mark.parametrize("T,Hkv", [(1, 1), (127, 2), (300, 4), (1000, 8)])
def test_split_contiguous(T, Hkv, A):
    k, v = random_kv(T, Hkv, seed=3000 + T)
    run_case(k, v, A)


@pytest.mark.parametrize("A", [2, 6])
@pytest.mark.parametrize("T,bt", [(700, 16), (513, 32), (129, 8)])
def test_split_paged(T, bt, A):
    k, v = random_kv(T, 2, seed=3100 + T)
    run_case(k, v, A, bt=bt, seed=T)


@pytest.mark.parametrize("A", [2, 6])
def test_split_llama3_8b_layer(A):
    w = inputs.WORKLOADS["llama3-8b-32k"]
    run_case(inputs.kv(w, "k", layer=3), inputs.kv(w, "v", layer=3), A)


def test_verify_over_codes_merged_from_2_plus_6():
    """The merged codes of a 2 + 6 split are the 4 + 4 codes, so verification
    over them gives the same output bit for bit."""
    T, Hkv, G, nq = 2048, 2, 4, 4
    k, v = random_kv(T, Hkv, seed=3300)
    codes26, meta26, L, tdev = run_case(k, v, 2)
    pool = lynx.KVPool.allocate(L, 1)
    pool.encode(0, T, tdev, k.cuda(), v.cuda())
    pool.merge()
    g = torch.Generator().manual_seed(5)
    q = torch.randn(1, nq, Hkv * G, 128, generator=g).to(torch.bfloat16).cuda()
    lens = torch.tensor([T], dtype=torch.int32, device="cuda")
    ws = lynx.workspace(L, 1, Hkv * G, nq, T)
    outs = []
    for kc, vc, m in ((codes26["k"], codes26["v"], meta26), (pool.k_codes, pool.v_codes, pool.meta)):
        o = torch.empty(1, nq, Hkv * G, 128, dtype=torch.bfloat16, device="cuda")
        lynx.lynx_attn_verify(L, 1, Hkv * G, nq, T, lens, tdev, kc, vc, m, q, None, None, o, ws)
        outs.append(o)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
