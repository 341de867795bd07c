"""GPU end to end: the split-stream transfer with real stream overlap.

Each layer's anchor planes are resident; its residual planes start in pinned
host memory and are copied to the device on a side stream (standing in for
the network transfer of the low-order half, Sec. 4).  The main stream runs
anchor decode for every layer while those copies are in flight, then waits
on each layer's copy event, merges that layer's planes back into 8-bit codes
and runs verification attention over them.  Every output is checked against
the CPU oracle on the same inputs, so a missing or misplaced wait (a merge
that reads a residual before its copy lands) shows as a parity failure.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests._util import LSE_ATOL, LSE_RTOL, assert_close
from tests.gpu_cases import bits, note, random_bf16, random_kv

pytestmark = pytest.mark.gpu


def _layer_inputs(lens, Hkv, layer):
    kv = [random_kv(T, Hkv, seed=7000 + 97 * layer + i) for i, T in enumerate(lens)]
    return [k for k, _ in kv], [v for _, v in kv]


@pytest.mark.parametrize("paged", [False, True])
def test_split_stream_pipeline(paged):
    layers, Hkv, G, nq = 3, 2, 4, 4
    Hq = G * Hkv
    lens = [700, 129, 33, 1]
    B, max_len = len(lens), max(lens)
    if paged:
        bt = 16
        table, n_blocks = inputs.paged_block_table(torch.tensor(lens), bt, 11)
    else:
        bt = max_len
        table, n_blocks = torch.arange(B, dtype=torch.int32).view(B, 1), B
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt, max_blocks_per_seq=table.shape[1],
                    num_blocks=n_blocks, max_tokens=max_len)
    OL = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=table.shape[1], max_tokens=max_len)
    tdev = table.cuda()
    lens_dev = torch.tensor(lens, dtype=torch.int32).cuda()

    # Producer side: encode every layer, then move the residual planes of the
    # whole cache to pinned host memory and clear them on the device.
    pools, whole = lynx.KVPool.allocate_layers(L, B, layers)
    ref_planes, ref_meta, qs = [], [], []
    for l in range(layers):
        ks, vs = _layer_inputs(lens, Hkv, l)
        for b in range(B):
            note(f"pipeline paged={paged} encode layer={l} b={b} T={lens[b]}")
            pools[l].encode(b, lens[b], tdev, ks[b].cuda(), vs[b].cuda())
        planes, meta = oracle.encode_batch(OL, lens, table.numpy(), [bits(k) for k in ks],
                                           [bits(v) for v in vs], n_blocks)
        ref_planes.append(planes)
        ref_meta.append(meta)
        qs.append((random_bf16((B, Hq, 128), seed=300 + l), random_bf16((B, nq, Hq, 128), seed=400 + l)))
    torch.cuda.synchronize()
    host = {}
    for name in ("k_res", "v_res"):
        host[name] = torch.empty(getattr(whole, name).numel(), dtype=torch.uint8, pin_memory=True)
        host[name].copy_(getattr(whole, name))
        getattr(whole, name).zero_()
    whole.k_codes.fill_(0xA5)
    whole.v_codes.fill_(0xA5)
    torch.cuda.synchronize()

    # Consumer side.  Every buffer used below is allocated before the side
    # stream starts and stays referenced until the final synchronisation.
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    dec_out = [torch.empty(B, Hq, 128, dtype=torch.bfloat16, device="cuda") for _ in range(layers)]
    dec_lse = [torch.empty(B, Hq, dtype=torch.float32, device="cuda") for _ in range(layers)]
    ver_out = [torch.empty(B, nq, Hq, 128, dtype=torch.bfloat16, device="cuda") for _ in range(layers)]
    ws_dec = lynx.workspace(L, B, Hq, 1, max_len)
    ws_ver = lynx.workspace(L, B, Hq, nq, max_len)
    qd = [(a.cuda(), b.cuda()) for a, b in qs]
    n = L.plane_bytes(64)
    arrived = [torch.cuda.Event() for _ in range(layers)]
    side.wait_stream(main)
    torch.cuda.synchronize()

    note(f"pipeline paged={paged} residual copies on the side stream")
    with torch.cuda.stream(side):
        for l in range(layers):
            for name in ("k_res", "v_res"):
                getattr(pools[l], name).copy_(host[name][l * n:(l + 1) * n], non_blocking=True)
            arrived[l].record(side)
    note(f"pipeline paged={paged} anchor decode of every layer on the main stream")
    for l in range(layers):
        lynx.lynx_attn_anchor_decode(L, B, Hq, max_len, lens_dev, tdev, pools[l].k_anc, pools[l].v_anc,
                                     pools[l].meta, qd[l][0], dec_out[l], dec_lse[l], ws_dec,
                                     stream=main)
    note(f"pipeline paged={paged} merge and verify per layer after its copy event")
    for l in range(layers):
        main.wait_event(arrived[l])
        pools[l].merge(stream=main)
        lynx.lynx_attn_verify(L, B, Hq, nq, max_len, lens_dev, tdev, pools[l].k_codes,
                              pools[l].v_codes, pools[l].meta, qd[l][1], None, None, ver_out[l],
                              ws_ver, stream=main)
    torch.cuda.synchronize()

    for l in range(layers):
        planes, meta = ref_planes[l], ref_meta[l]
        q1, qk = qs[l]
        kc = oracle.merge(planes["k_anc"], planes["k_res"])
        vc = oracle.merge(planes["v_anc"], planes["v_res"])
        assert np.array_equal(pools[l].k_codes.cpu().numpy(), kc), f"layer {l}: K codes differ"
        assert np.array_equal(pools[l].v_codes.cpu().numpy(), vc), f"layer {l}: V codes differ"
        ref, ref_lse = oracle.anchor_decode(OL, Hq, np.array(lens), table.numpy(), planes["k_anc"],
                                            planes["v_anc"], meta, bits(q1))
        assert_close(dec_out[l].float().cpu().numpy(), ref, what=f"pipeline decode layer {l}")
        np.testing.assert_allclose(dec_lse[l].cpu().numpy(), ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)
        vref, _ = oracle.verify(OL, Hq, np.array(lens), table.numpy(), kc, vc, meta, bits(qk), None, None)
        assert_close(ver_out[l].float().cpu().numpy(), vref, what=f"pipeline verify layer {l}")


@pytest.mark.parametrize("variant", ["biased", "centred"])
def test_hier_split_stream_pipeline(variant):
    """The hierarchical codec of Alg. 1 on the same split-stream schedule: the
    anchor-only BF16 reconstruction runs on the main stream while the
    correction planes are copied from pinned host memory on a side stream;
    the merge and the full reconstruction wait on the copy event.  Every
    plane and output is checked bit for bit against the oracle."""
    T, Hkv, bt, alpha = 1500, 2, 16, 20.0
    vid = oracle.H_VARIANTS[variant]
    k, v = random_kv(T, Hkv, seed=7500 + vid)
    table, n_blocks = inputs.paged_block_table(torch.tensor([T]), bt, 17)
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt, max_blocks_per_seq=table.shape[1],
                    num_blocks=n_blocks, max_tokens=T)
    OL = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=table.shape[1], max_tokens=T)
    pool = lynx.KVPool.allocate(L, 1)
    hm = lynx.HMeta.empty(L, 1)
    tdev = table.cuda()
    note(f"hier pipeline variant={variant} encode T={T}")
    lynx.lynx_hkv_encode(L, 0, T, tdev, k.cuda(), v.cuda(), alpha, vid, pool.k_anc, pool.v_anc,
                         pool.k_res, pool.v_res, hm)
    torch.cuda.synchronize()
    host = {}
    for name in ("k_res", "v_res"):
        host[name] = torch.empty(getattr(pool, name).numel(), dtype=torch.uint8, pin_memory=True)
        host[name].copy_(getattr(pool, name))
        getattr(pool, name).zero_()
    pool.k_codes.fill_(0xA5)
    pool.v_codes.fill_(0xA5)
    outs = {m: (torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device="cuda"),
                torch.empty(T, Hkv, 128, dtype=torch.bfloat16, device="cuda")) for m in ("anchor", "full")}
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    arrived = torch.cuda.Event()
    side.wait_stream(main)
    torch.cuda.synchronize()

    note(f"hier pipeline variant={variant} correction copies on the side stream, anchor dequant on main")
    with torch.cuda.stream(side):
        pool.k_res.copy_(host["k_res"], non_blocking=True)
        pool.v_res.copy_(host["v_res"], non_blocking=True)
        arrived.record(side)
    lynx.lynx_hkv_dequant(L, 0, T, tdev, False, pool.k_anc, pool.v_anc, alpha, vid, hm, *outs["anchor"],
                          stream=main)
    main.wait_event(arrived)
    pool.merge(stream=main)
    lynx.lynx_hkv_dequant(L, 0, T, tdev, True, pool.k_codes, pool.v_codes, alpha, vid, hm, *outs["full"],
                          stream=main)
    torch.cuda.synchronize()

    nbytes = oracle.plane_bytes(OL, n_blocks, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    ohm = oracle.HMeta.empty(OL, 1)
    oracle.hencode(OL, 0, T, table.numpy(), bits(k), bits(v), alpha, planes, ohm, variant)
    codes = {p: oracle.merge(planes[p + "_anc"], planes[p + "_res"]) for p in ("k", "v")}
    assert np.array_equal(pool.k_codes.cpu().numpy(), codes["k"]), "K codes differ"
    assert np.array_equal(pool.v_codes.cpu().numpy(), codes["v"]), "V codes differ"
    ref = {"anchor": oracle.hdequant("anchor", OL, 0, T, table.numpy(), planes["k_anc"], planes["v_anc"],
                                     alpha, ohm, variant),
           "full": oracle.hdequant("full", OL, 0, T, table.numpy(), codes["k"], codes["v"], alpha, ohm,
                                   variant)}
    for mode in ("anchor", "full"):
        for i, name in enumerate(("K", "V")):
            got, want = bits(outs[mode][i]), ref[mode][i]
            assert np.array_equal(got, want), f"{mode} {name}: {np.count_nonzero(got != want)} values differ"
