"""GPU parity at the full sizes of the five workloads (paper-shaped synthetic
inputs from paper_2607_01831_amd.inputs), in the launch configurations the
benchmark uses.

The codec (planes, metadata, merged codes) is compared bit for bit over the
whole workload.  Attention outputs are compared on sampled (sequence, kv head)
units, which the oracle computes one by one (unit_mask); the tolerance is the
elementwise 2e-2 + 1e-2 |ref| against the fp64 oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests._util import LSE_ATOL, LSE_RTOL, assert_close
from tests.gpu_cases import bits, build_cache, note, random_bf16, random_kv

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def assert_planes_equal(c):
    for name in ("k_anc", "v_anc", "k_res", "v_res"):
        got = getattr(c.pool, name).cpu().numpy()
        assert np.array_equal(got, c.planes[name]), f"{name}: {np.count_nonzero(got != c.planes[name])} bytes differ"
    m = c.pool.meta
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        got = getattr(m, name).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), getattr(c.meta, name).view(np.uint32)), name


def assert_codes_equal(c):
    assert np.array_equal(c.pool.k_codes.cpu().numpy(), oracle.merge(c.planes["k_anc"], c.planes["k_res"]))
    assert np.array_equal(c.pool.v_codes.cpu().numpy(), oracle.merge(c.planes["v_anc"], c.planes["v_res"]))


def sample_units(B, Hkv, n, seed):
    rng = np.random.default_rng(seed)
    mask = np.zeros((B, Hkv), np.uint8)
    for u in rng.choice(B * Hkv, size=min(n, B * Hkv), replace=False):
        mask[u // Hkv, u % Hkv] = 1
    return mask


def check_units(out, ref, mask, G, what, lse=None, ref_lse=None):
    """Compare the heads of every unit (b, h) selected by mask; out/ref are
    [B][..][Hq][128] with the head axis second to last."""
    for b, h in zip(*np.nonzero(mask)):
        sl = (b, Ellipsis, slice(h * G, (h + 1) * G), slice(None))
        assert_close(out[sl], ref[sl], what=f"{what} b={b} h={h}")
        if lse is not None:
            np.testing.assert_allclose(lse[b, ..., h * G:(h + 1) * G], ref_lse[b, ..., h * G:(h + 1) * G],
                                       rtol=LSE_RTOL, atol=LSE_ATOL)


def run_decode(c, q, with_lse=True):
    B, Hq = c.B, q.shape[1]
    out = torch.empty(B, Hq, 128, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, Hq, dtype=torch.float32, device="cuda") if with_lse else None
    max_len = max(c.lens)
    ws = lynx.workspace(c.L, B, Hq, 1, max_len)
    note(f"full-size anchor decode B={B} Hq={Hq} max_len={max_len}")
    lynx.lynx_attn_anchor_decode(c.L, B, Hq, max_len, c.lens_dev(), c.table_dev(), c.pool.k_anc,
                                 c.pool.v_anc, c.pool.meta, q.cuda(), out, lse, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), (lse.cpu().numpy() if with_lse else None)


def run_verify(c, q, kn, vn):
    B, nq, Hq = c.B, q.shape[1], q.shape[2]
    out = torch.empty(B, nq, Hq, 128, dtype=torch.bfloat16, device="cuda")
    max_len = max(c.lens)
    ws = lynx.workspace(c.L, B, Hq, nq, max_len)
    note(f"full-size verify B={B} k={nq} Hq={Hq} max_len={max_len}")
    lynx.lynx_attn_verify(c.L, B, Hq, nq, max_len, c.lens_dev(), c.table_dev(), c.pool.k_codes,
                          c.pool.v_codes, c.pool.meta, q.cuda(),
                          None if kn is None else kn.cuda(), None if vn is None else vn.cuda(), out, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


def oracle_decode(c, q, mask):
    return oracle.anchor_decode(c.OL, q.shape[1], np.array(c.lens), c.table.numpy(), c.planes["k_anc"],
                                c.planes["v_anc"], c.meta, bits(q), unit_mask=mask)


def oracle_verify(c, q, kn, vn, mask):
    kc = oracle.merge(c.planes["k_anc"], c.planes["k_res"])
    vc = oracle.merge(c.planes["v_anc"], c.planes["v_res"])
    out, _ = oracle.verify(c.OL, q.shape[2], np.array(c.lens), c.table.numpy(), kc, vc, c.meta,
                           bits(q), None if kn is None else bits(kn), None if vn is None else bits(vn),
                           unit_mask=mask)
    return out


def vnmse(o_hat, o):
    """E ||o_hat - o||^2 / ||o||^2 over the rows of [..][128] arrays."""
    o_hat = np.asarray(o_hat, np.float64).reshape(-1, 128)
    o = np.asarray(o, np.float64).reshape(-1, 128)
    return float((((o_hat - o) ** 2).sum(axis=1) / (o ** 2).sum(axis=1)).mean())


def test_llama3_8b_32k_layer():
    """One layer of the benchmark workload (32 q / 8 kv heads, 32K context):
    codec bit-exact; decode and verify (k = 8 with the draft tail) on every
    kv head."""
    w = inputs.WORKLOADS["llama3-8b-32k"]
    layer = 5
    k = inputs.kv(w, "k", layer=layer)
    v = inputs.kv(w, "v", layer=layer)
    c = build_cache([k], [v], w.Hkv)
    assert_planes_equal(c)
    assert_codes_equal(c)
    mask = np.ones((1, w.Hkv), np.uint8)
    q = inputs.queries(w, layer=layer)
    out, lse = run_decode(c, q)
    ref, ref_lse = oracle_decode(c, q, mask)
    check_units(out, ref, mask, w.G, "32K decode", lse, ref_lse)
    qv = inputs.queries(w, layer=layer, step=1, nq=w.drafts)
    kn, vn = inputs.drafts_kv(w, layer=layer)
    outv = run_verify(c, qv, kn, vn)
    refv = oracle_verify(c, qv, kn, vn, mask)
    check_units(outv, refv, mask, w.G, "32K verify k=8")


def test_verify_128k():
    """Verification at 128K context, k = 8 drafts with the causal draft tail:
    codec and merge bit-exact over the layer; verify on 3 sampled kv heads."""
    w = inputs.WORKLOADS["llama3-8b-verify-128k"]
    k = inputs.kv(w, "k")
    v = inputs.kv(w, "v")
    c = build_cache([k], [v], w.Hkv)
    del k, v
    assert_planes_equal(c)
    assert_codes_equal(c)
    mask = sample_units(1, w.Hkv, 3, seed=31)
    qv = inputs.queries(w, nq=w.drafts)
    kn, vn = inputs.drafts_kv(w)
    outv = run_verify(c, qv, kn, vn)
    refv = oracle_verify(c, qv, kn, vn, mask)
    check_units(outv, refv, mask, w.G, "128K verify k=8")
    # the anchor-only decode of draft 0 and the verification of draft 0 over
    # the merged codes (no tail), each against the oracle; then how far the
    # anchor-only output is from the full one (what the residual removes),
    # on the GPU and in the oracle
    q0 = qv[:, 0].contiguous()
    out_a, _ = run_decode(c, q0, with_lse=False)
    ref_a, _ = oracle_decode(c, q0, mask)
    check_units(out_a, ref_a, mask, w.G, "128K anchor decode of draft 0")
    q0v = q0.view(1, 1, w.Hq, 128)
    out_f = run_verify(c, q0v, None, None)[:, 0]
    ref_f = oracle_verify(c, q0v, None, None, mask)[:, 0]
    check_units(out_f, ref_f, mask, w.G, "128K verify of draft 0, no tail")
    heads = [hh for h in np.nonzero(mask[0])[0] for hh in range(h * w.G, (h + 1) * w.G)]
    dev_gpu = vnmse(out_a[0, heads], out_f[0, heads])
    dev_ref = vnmse(ref_a[0, heads], ref_f[0, heads])
    note(f"128K anchor-only vs full, draft 0: vNMSE {dev_gpu:.4g} (oracle {dev_ref:.4g})")
    assert dev_ref > 0
    assert abs(dev_gpu - dev_ref) <= 0.1 * dev_ref


def test_paged_b16_decode():
    """Batched paged anchor decode: 16 sequences of 16K..64K tokens in
    16-token blocks under a random block table; codec bit-exact over the
    pool, decode on 8 sampled (sequence, kv head) units."""
    w = inputs.WORKLOADS["paged-b16-16k-64k"]
    lens = inputs.seq_lengths(w).tolist()
    ks = [inputs.kv(w, "k", seq=b, T=T) for b, T in enumerate(lens)]
    vs = [inputs.kv(w, "v", seq=b, T=T) for b, T in enumerate(lens)]
    c = build_cache(ks, vs, w.Hkv, bt=w.block_tokens, seed=inputs.seed_of(w.wid, inputs.T_BLOCKS),
                    merge=False, max_tokens=w.context)
    del ks, vs
    assert_planes_equal(c)
    mask = sample_units(w.batch, w.Hkv, 8, seed=41)
    q = inputs.queries(w)
    out, lse = run_decode(c, q)
    ref, ref_lse = oracle_decode(c, q, mask)
    check_units(out, ref, mask, w.G, "paged decode", lse, ref_lse)


def test_70b_b4_128k():
    """70B-shaped batch: 4 x 128K, 64 q / 8 kv heads (G = 8).  Codec and merge
    bit-exact; two decode steps, then verify k = 4 with the draft tail, each on
    3 sampled units."""
    w = inputs.WORKLOADS["70b-overlap-b4-128k"]
    ks = [inputs.kv(w, "k", seq=b) for b in range(w.batch)]
    vs = [inputs.kv(w, "v", seq=b) for b in range(w.batch)]
    c = build_cache(ks, vs, w.Hkv)
    del ks, vs
    assert_planes_equal(c)
    assert_codes_equal(c)
    for step in (0, w.decode_steps - 1):
        mask = sample_units(w.batch, w.Hkv, 3, seed=50 + step)
        q = inputs.queries(w, step=step)
        out, lse = run_decode(c, q)
        ref, ref_lse = oracle_decode(c, q, mask)
        check_units(out, ref, mask, w.G, f"70B decode step {step}", lse, ref_lse)
    mask = sample_units(w.batch, w.Hkv, 3, seed=59)
    qv = inputs.queries(w, step=w.decode_steps, nq=w.drafts)
    kn, vn = inputs.drafts_kv(w)
    outv = run_verify(c, qv, kn, vn)
    refv = oracle_verify(c, qv, kn, vn, mask)
    check_units(outv, refv, mask, w.G, "70B verify k=4")


def test_one_round_long_splits():
    """A contiguous batch large enough that one round of workgroups (two per
    CU) needs 4096-token splits: 512K tokens, 4 kv heads, G = 4.  Decode (its
    split merge in the same launch) and verification of k = 4 drafts with
    their tail (16 query rows per workgroup), 2 sampled units each against
    the oracle."""
    Hkv, G, T, nq = 4, 4, 524288, 4
    k, v = random_kv(T, Hkv, seed=6100)
    c = build_cache([k], [v], Hkv)
    del k, v
    q = random_bf16((1, Hkv * G, 128), seed=6101)
    out, lse = run_decode(c, q)
    mask = sample_units(1, Hkv, 2, seed=6102)
    ref, ref_lse = oracle_decode(c, q, mask)
    check_units(out, ref, mask, G, "one-round decode over 512K tokens", lse, ref_lse)
    qv = random_bf16((1, nq, Hkv * G, 128), seed=6103)
    kn = random_bf16((1, nq, Hkv, 128), seed=6104)
    vn = random_bf16((1, nq, Hkv, 128), seed=6105)
    outv = run_verify(c, qv, kn, vn)
    mask = sample_units(1, Hkv, 2, seed=6106)
    refv = oracle_verify(c, qv, kn, vn, mask)
    check_units(outv, refv, mask, G, "one-round verification over 512K tokens")
