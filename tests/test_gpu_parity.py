"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.

Codec and packed layouts must match bit for bit; attention outputs (BF16)
must satisfy |gpu - ref| <= 2e-2 + 1e-2 |ref| elementwise against the fp64
oracle.  Sizes span several 128-token groups and ragged tails; edge cases
cover one-token and empty sequences, constant groups, signed zeros,
denormals, G = 1..8 and k = 1..64.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests._util import LSE_ATOL, LSE_RTOL, assert_close
from tests.gpu_cases import (bits, build_cache, gpu_anchor_decode, gpu_verify, note, random_bf16,
                             random_kv)

pytestmark = pytest.mark.gpu


def assert_codec_equal(c):
    for name in ("k_anc", "v_anc", "k_res", "v_res"):
        got = getattr(c.pool, name).cpu().numpy()
        assert np.array_equal(got, c.planes[name]), f"{name}: {np.count_nonzero(got != c.planes[name])} bytes differ"
    m = c.pool.meta
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        got = getattr(m, name).cpu().numpy()
        ref = getattr(c.meta, name)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), f"{name} differs"


# ------------------------------------------------------------------ codec --

@pytest.mark.parametrize("T", [1, 15, 16, 17, 127, 128, 129, 300, 1000])
@pytest.mark.parametrize("Hkv", [1, 4])
def test_encode_bit_exact_contiguous(T, Hkv):
    k, v = random_kv(T, Hkv, seed=T * 10 + Hkv)
    c = build_cache([k], [v], Hkv, merge=False)
    assert_codec_equal(c)


def test_encode_bit_exact_paged_ragged():
    lens = [37, 300, 129, 1, 16]
    kv = [random_kv(T, 2, seed=100 + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], 2, bt=16, seed=5, merge=False,
                    max_tokens=320)
    assert_codec_equal(c)


def test_encode_adversarial_groups():
    """Constant groups, two-valued groups, +-0, denormals, huge values and exact
    rounding ties decide the same codes on both sides."""
    T, Hkv = 260, 2
    g = torch.Generator().manual_seed(3)
    x = torch.randn(T, Hkv, 128, generator=g)
    x[:, 0, 0] = 3.25                                   # constant K column
    x[:, 0, 1] = torch.where(torch.arange(T) % 3 == 0, -7.0, 9.0)
    x[:, 0, 2] = -0.0
    x[:, 0, 3] = torch.randn(T, generator=g) * 1e-39     # denormals
    x[:, 1, 4] = torch.randn(T, generator=g) * 1e37      # huge
    x[:, 1, 5] = torch.arange(T) % 256                   # integers: scale 1, ties
    v = torch.randn(T, Hkv, 128, generator=g)
    v[0] = 1.5                                           # constant V rows
    v[1, :, :64] = -0.0
    v[1, :, 64:] = 0.0
    v[2, :, :4] = torch.tensor([0.0, 255.0, 126.5, 2.5]) # half-even ties
    v[2, :, 4:] = 0.0
    v[3] = torch.randn(Hkv, 128, generator=g) * 1e-38
    c = build_cache([x.to(torch.bfloat16)], [v.to(torch.bfloat16)], Hkv, merge=False)
    assert_codec_equal(c)


# sizes around the kernel's 8-byte pieces and its 1 KB wave rounds, and one
# past the 8192 workgroups x 4 waves x 1 KB of one grid round (so waves loop)
# with a ragged tail
@pytest.mark.parametrize("n", [1, 7, 8, 9, 15, 16, 17, 1023, 1024, 1025, 4096, 4096 + 5, 1 << 20,
                               (32 << 20) + 3 * 1024 + 8 * 5 + 5])
def test_merge_bit_exact(n):
    g = torch.Generator().manual_seed(n)
    a = torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8)
    r = torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8)
    codes = torch.full((2 * n,), 0xA5, dtype=torch.uint8, device="cuda")
    note(f"merge n={n}")
    lynx.lynx_kv_merge(a.cuda(), r.cuda(), codes)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), oracle.merge(a.numpy(), r.numpy()))


@pytest.mark.parametrize("offs", [(16, 48, 32), (4096 + 16, 16, 4096 + 48)])
def test_merge_at_16_byte_offsets(offs):
    """Planes and codes that start 16 bytes past an allocation's alignment (the
    ABI asks for 16): the 8-byte loads and 16-byte stores of the merge stay
    exact, and nothing outside the codes is written."""
    oa, orr, oc = offs
    n = 3 * 1024 + 8 * 3 + 5
    g = torch.Generator().manual_seed(oa + orr)
    a = torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8)
    r = torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8)
    abuf = torch.zeros(oa + n + 64, dtype=torch.uint8, device="cuda")
    rbuf = torch.zeros(orr + n + 64, dtype=torch.uint8, device="cuda")
    cbuf = torch.full((oc + 2 * n + 64,), 0xA5, dtype=torch.uint8, device="cuda")
    abuf[oa:oa + n] = a.cuda()
    rbuf[orr:orr + n] = r.cuda()
    note(f"merge n={n} offsets={offs}")
    lynx.lynx_kv_merge(abuf[oa:oa + n], rbuf[orr:orr + n], cbuf[oc:oc + 2 * n])
    torch.cuda.synchronize()
    got = cbuf.cpu().numpy()
    assert np.array_equal(got[oc:oc + 2 * n], oracle.merge(a.numpy(), r.numpy()))
    assert (got[:oc] == 0xA5).all() and (got[oc + 2 * n:] == 0xA5).all()


def test_merge_of_encoded_planes():
    k, v = random_kv(640, 4, seed=9)
    c = build_cache([k], [v], 4)
    assert np.array_equal(c.pool.k_codes.cpu().numpy(), oracle.merge(c.planes["k_anc"], c.planes["k_res"]))
    assert np.array_equal(c.pool.v_codes.cpu().numpy(), oracle.merge(c.planes["v_anc"], c.planes["v_res"]))


# -------------------------------------------------------------- attention --

def oracle_decode(c, q, unit_mask=None):
    return oracle.anchor_decode(c.OL, q.shape[1], np.array(c.lens), c.table.numpy(),
                                c.planes["k_anc"], c.planes["v_anc"], c.meta, bits(q),
                                unit_mask=unit_mask)


def oracle_verify(c, q, k_new=None, v_new=None, unit_mask=None):
    kc = oracle.merge(c.planes["k_anc"], c.planes["k_res"])
    vc = oracle.merge(c.planes["v_anc"], c.planes["v_res"])
    return oracle.verify(c.OL, q.shape[2], np.array(c.lens), c.table.numpy(), kc, vc, c.meta,
                         bits(q), None if k_new is None else bits(k_new),
                         None if v_new is None else bits(v_new), unit_mask=unit_mask)


@pytest.mark.parametrize("G", [1, 2, 4, 8])
@pytest.mark.parametrize("T", [1, 17, 300, 1500])
def test_anchor_decode(G, T):
    Hkv = 2
    k, v = random_kv(T, Hkv, seed=G * 1000 + T)
    c = build_cache([k], [v], Hkv, merge=False)
    q = random_bf16((1, G * Hkv, 128), seed=T + G)
    out, lse = gpu_anchor_decode(c, q)
    ref, ref_lse = oracle_decode(c, q)
    assert_close(out, ref, what=f"anchor decode G={G} T={T}")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_anchor_decode_paged_ragged_batch():
    lens = [700, 33, 1, 1024, 129]
    kv = [random_kv(T, 2, seed=200 + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], 2, bt=16, seed=7, merge=False)
    q = random_bf16((len(lens), 8, 128), seed=77)
    out, lse = gpu_anchor_decode(c, q)
    ref, ref_lse = oracle_decode(c, q)
    assert_close(out, ref, what="paged ragged decode")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_anchor_decode_empty_sequence():
    lens = [0, 50]
    kv = [random_kv(max(T, 1), 1, seed=300 + i) for i, T in enumerate(lens)]
    ks = [kv[0][0][:0], kv[1][0]]
    vs = [kv[0][1][:0], kv[1][1]]
    c = build_cache(ks, vs, 1, merge=False)
    q = random_bf16((2, 2, 128), seed=1)
    out, lse = gpu_anchor_decode(c, q)
    assert (out[0] == 0).all() and np.isneginf(lse[0]).all()
    ref, _ = oracle_decode(c, q)
    assert_close(out[1], ref[1], what="second sequence")


@pytest.mark.parametrize("nq,tail", [(1, False), (1, True), (4, True), (8, True), (8, False), (64, True)])
def test_verify(nq, tail):
    Hkv, G = 2, 4
    lens = [300, 129]
    kv = [random_kv(T, Hkv, seed=400 + i + nq) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv)
    q = random_bf16((2, nq, Hkv * G, 128), seed=nq)
    kn = random_bf16((2, nq, Hkv, 128), seed=nq + 1) if tail else None
    vn = random_bf16((2, nq, Hkv, 128), seed=nq + 2) if tail else None
    out = gpu_verify(c, q, kn, vn)
    ref, _ = oracle_verify(c, q, kn, vn)
    assert_close(out, ref, what=f"verify k={nq} tail={tail}")


@pytest.mark.parametrize("bt", [16, 8])
def test_verify_paged_ragged(bt):
    """Verification over paged pools with ragged lengths: block_tokens 16
    (16-token runs share a block) and 8 (every token row is looked up on its
    own), k = 8 drafts with the causal tail, 32 query rows per kv head."""
    Hkv, G, nq = 2, 4, 8
    lens = [1000, 37, 513]
    kv = [random_kv(T, Hkv, seed=800 + bt + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, bt=bt, seed=bt)
    q = random_bf16((len(lens), nq, Hkv * G, 128), seed=810 + bt)
    kn = random_bf16((len(lens), nq, Hkv, 128), seed=811 + bt)
    vn = random_bf16((len(lens), nq, Hkv, 128), seed=812 + bt)
    out = gpu_verify(c, q, kn, vn)
    ref, _ = oracle_verify(c, q, kn, vn)
    assert_close(out, ref, what=f"paged verify bt={bt}")


@pytest.mark.parametrize("boost", [30.0, 400.0])
def test_verify_dominant_late_token(boost):
    """One draft row meets a late context token whose score dwarfs the rest:
    with boost 400 the fixed softmax reference of the first tile overflows and
    the wavefronts holding that token redo their tiles with a running maximum;
    boost 30 stays on the fast path."""
    T, Hkv, G, nq = 3000, 2, 4, 8
    g = torch.Generator().manual_seed(900 + int(boost))
    q = torch.randn(1, nq, G * Hkv, 128, generator=g)
    k = torch.randn(T, Hkv, 128, generator=g)
    v = torch.randn(T, Hkv, 128, generator=g)
    for h in range(Hkv):
        k[2500, h] = boost * q[0, 3, h * G] / q[0, 3, h * G].norm()
    c = build_cache([k.to(torch.bfloat16)], [v.to(torch.bfloat16)], Hkv)
    qb = q.to(torch.bfloat16)
    kn = random_bf16((1, nq, Hkv, 128), seed=901)
    vn = random_bf16((1, nq, Hkv, 128), seed=902)
    out = gpu_verify(c, qb, kn, vn)
    ref, _ = oracle_verify(c, qb, kn, vn)
    assert_close(out, ref, what=f"verify dominant token x{boost}")


@pytest.mark.slow
def test_verify_eight_group_splits():
    """64K context x 8 kv heads, k = 8: the plan picks 1024-token splits (8
    groups, two per wavefront); 2 sampled kv heads against the oracle."""
    T, Hkv, G, nq = 65536, 8, 4, 8
    k, v = random_kv(T, Hkv, seed=950)
    c = build_cache([k], [v], Hkv)
    q = random_bf16((1, nq, Hkv * G, 128), seed=951)
    kn = random_bf16((1, nq, Hkv, 128), seed=952)
    vn = random_bf16((1, nq, Hkv, 128), seed=953)
    mask = np.zeros((1, Hkv), np.uint8)
    mask[0, [2, 7]] = 1
    out = gpu_verify(c, q, kn, vn)
    ref, _ = oracle_verify(c, q, kn, vn, unit_mask=mask)
    for h in (2, 7):
        sl = (0, slice(None), slice(h * G, (h + 1) * G), slice(None))
        assert_close(out[sl], ref[sl], what=f"64K verify kv head {h}")


def test_tiny_config_end_to_end():
    """Tiny workload: 1 layer, 8 q / 4 kv heads, 4096 tokens, 4 K outlier
    channels x10 per kv head; encode, merge, anchor decode, verify k = 1."""
    w = inputs.WORKLOADS["tiny-gqa2-4k"]
    k = inputs.kv(w, "k")
    v = inputs.kv(w, "v")
    c = build_cache([k], [v], w.Hkv)
    assert_codec_equal(c)
    assert np.array_equal(c.pool.k_codes.cpu().numpy(), oracle.merge(c.planes["k_anc"], c.planes["k_res"]))
    q = inputs.queries(w)
    out, lse = gpu_anchor_decode(c, q)
    ref, ref_lse = oracle_decode(c, q)
    assert_close(out, ref, what="tiny anchor decode")
    qv = inputs.queries(w, nq=1).view(1, 1, w.Hq, 128)
    outv = gpu_verify(c, qv)
    refv, _ = oracle_verify(c, qv)
    assert_close(outv, refv, what="tiny verify")


@pytest.mark.parametrize("boost", [30.0, 400.0])
def test_anchor_decode_dominant_late_token(boost):
    """A late token whose score dwarfs every earlier one: exercises the
    kernel's fallback that rescales when the first tile's maximum is far too
    small a reference (boost 400 overflows it, boost 30 does not)."""
    T, Hkv, G = 3000, 2, 4
    g = torch.Generator().manual_seed(int(boost))
    q = torch.randn(1, G * Hkv, 128, generator=g)
    k = torch.randn(T, Hkv, 128, generator=g)
    v = torch.randn(T, Hkv, 128, generator=g)
    for h in range(Hkv):
        k[2500, h] = boost * q[0, h * G] / q[0, h * G].norm()
    c = build_cache([k.to(torch.bfloat16)], [v.to(torch.bfloat16)], Hkv, merge=False)
    qb = q.to(torch.bfloat16)
    out, lse = gpu_anchor_decode(c, qb)
    ref, ref_lse = oracle_decode(c, qb)
    assert_close(out, ref, what=f"dominant token x{boost}")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_anchor_decode_workspace_reuse():
    """Back-to-back decode calls of different shapes share one workspace;
    each call's result must not depend on what the previous one left there."""
    Hkv, G = 2, 4
    ca = build_cache(*map(list, zip(*[random_kv(T, Hkv, seed=500 + T) for T in (700, 5, 1500)])),
                     Hkv, merge=False)
    cb = build_cache(*map(list, zip(*[random_kv(T, Hkv, seed=600 + T) for T in (40, 2000)])),
                     Hkv, merge=False)
    nbytes = max(lynx.lynx_attn_workspace_bytes(c.L, c.B, Hkv * G, 1, max(c.lens)) for c in (ca, cb))
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    for rep, c in enumerate((ca, cb, ca, cb)):
        q = random_bf16((c.B, Hkv * G, 128), seed=rep % 2)
        out = torch.empty(c.B, Hkv * G, 128, dtype=torch.bfloat16, device="cuda")
        note(f"workspace reuse call {rep} lens={c.lens}")
        lynx.lynx_attn_anchor_decode(c.L, c.B, Hkv * G, max(c.lens), c.lens_dev(), c.table_dev(),
                                     c.pool.k_anc, c.pool.v_anc, c.pool.meta, q.cuda(), out, None, ws)
        torch.cuda.synchronize()
        ref, _ = oracle_decode(c, q)
        assert_close(out.float().cpu().numpy(), ref, what=f"reuse call {rep}")


def test_anchor_decode_many_units():
    """A wide batch of short sequences: 257 sequences x 64 kv heads, one
    split each."""
    Hkv, B = 64, 257
    g = torch.Generator().manual_seed(11)
    lens = torch.randint(1, 40, (B,), generator=g).tolist()
    kv = [random_kv(T, Hkv, seed=700 + i, outlier_cols=0) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, merge=False)
    q = random_bf16((B, Hkv, 128), seed=12)
    out, lse = gpu_anchor_decode(c, q)
    ref, ref_lse = oracle_decode(c, q)
    assert_close(out, ref, what="many units")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_anchor_decode_ragged_batch_stale_workspace():
    """A ragged batch over a workspace full of stale values: splits past a
    short sequence's end must not contribute."""
    Hkv, G = 8, 4
    lens = [6000, 100, 3000, 20, 5999, 1, 2500, 4097]
    kv = [random_kv(T, Hkv, seed=800 + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, merge=False)
    B, Hq = len(lens), Hkv * G
    q = random_bf16((B, Hq, 128), seed=13)
    n = lynx.lynx_attn_workspace_bytes(c.L, B, Hq, 1, max(lens))
    # partials filled with plausible-looking values (0x3F3F3F3F ~ 0.75); the
    # arrival counters at the head zeroed, as the header requires
    ws = torch.full((n,), 0x3F, dtype=torch.uint8, device="cuda")
    ws[:lynx.ATTN_COUNTER_BYTES].zero_()
    out = torch.empty(B, Hq, 128, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, Hq, dtype=torch.float32, device="cuda")
    note(f"ragged stale workspace lens={lens}")
    lynx.lynx_attn_anchor_decode(c.L, B, Hq, max(lens), c.lens_dev(), c.table_dev(), c.pool.k_anc,
                                 c.pool.v_anc, c.pool.meta, q.cuda(), out, lse, ws)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_decode(c, q)
    assert_close(out.float().cpu().numpy(), ref, what="ragged batch, stale workspace")
    np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_attention_calls_share_one_workspace():
    """Decode calls of different batch shapes, a decode with a BF16 tail (the
    combine kernel) and a verification pass take turns on one workspace: each
    call leaves the arrival counters at its head zero for the next."""
    Hkv, G = 4, 4
    Hq = Hkv * G
    lens = [3000, 700, 5000]
    kv = [random_kv(T, Hkv, seed=900 + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, merge=True)
    B = len(lens)
    nq = 3
    ws = lynx.workspace(c.L, B, Hq, nq, max(lens))
    q = random_bf16((B, Hq, 128), seed=21)
    qv = random_bf16((B, nq, Hq, 128), seed=22)
    kn = random_bf16((B, nq, Hkv, 128), seed=23)
    vn = random_bf16((B, nq, Hkv, 128), seed=24)
    ref, ref_lse = oracle_decode(c, q)
    ref_v, _ = oracle_verify(c, qv, kn, vn)
    for rep in range(3):
        note(f"shared workspace rep {rep}")
        out = torch.empty(B, Hq, 128, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(B, Hq, dtype=torch.float32, device="cuda")
        lynx.lynx_attn_anchor_decode(c.L, B, Hq, max(lens), c.lens_dev(), c.table_dev(),
                                     c.pool.k_anc, c.pool.v_anc, c.pool.meta, q.cuda(), out, lse, ws)
        # the first sequence alone (a smaller batch over the same counters)
        out1 = torch.empty(1, Hq, 128, dtype=torch.bfloat16, device="cuda")
        lynx.lynx_attn_anchor_decode(c.L, 1, Hq, lens[0], c.lens_dev()[:1], c.table_dev()[:1],
                                     c.pool.k_anc, c.pool.v_anc, c.pool.meta, q[:1].cuda(), out1,
                                     None, ws)
        outv = torch.empty(B, nq, Hq, 128, dtype=torch.bfloat16, device="cuda")
        lynx.lynx_attn_verify(c.L, B, Hq, nq, max(lens), c.lens_dev(), c.table_dev(),
                              c.pool.k_codes, c.pool.v_codes, c.pool.meta, qv.cuda(), kn.cuda(),
                              vn.cuda(), outv, ws)
        torch.cuda.synchronize()
        assert_close(out.float().cpu().numpy(), ref, what=f"decode rep {rep}")
        np.testing.assert_allclose(lse.cpu().numpy(), ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)
        assert_close(out1.float().cpu().numpy(), ref[:1], what=f"decode b=0 rep {rep}")
        assert_close(outv.float().cpu().numpy(), ref_v, what=f"verify rep {rep}")
    assert int(ws[:lynx.ATTN_COUNTER_BYTES].count_nonzero().item()) == 0


def _dominant(k, q, t, h, G, boost):
    """Make token t of kv head h score boost x |q| for the first query head of
    h's group; q is one sequence's [Hq][128] queries."""
    qh = q[h * G].float()
    k[t, h] = (boost * qh / qh.norm()).to(k.dtype)


def _decode_check_sampled(c, q, mask, what):
    out, lse = gpu_anchor_decode(c, q)
    ref, ref_lse = oracle_decode(c, q, unit_mask=mask)
    G = q.shape[1] // c.Hkv
    for b, h in zip(*np.nonzero(mask)):
        assert_close(out[b, h * G:(h + 1) * G], ref[b, h * G:(h + 1) * G], what=f"{what} b={b} h={h}")
        np.testing.assert_allclose(lse[b, h * G:(h + 1) * G], ref_lse[b, h * G:(h + 1) * G],
                                   rtol=LSE_RTOL, atol=LSE_ATOL)


@pytest.mark.slow
def test_anchor_decode_two_round_splits_dominant_token():
    """Splits of 8 groups (two rounds of the rolling fold): 2 x 32 kv heads x
    ~20K tokens.  One unit holds a token whose score overflows the first
    tile's reference (the workgroup redoes the split with a running maximum),
    one a milder outlier."""
    Hkv, G, lens = 32, 4, [20000, 19000]
    q = random_bf16((2, Hkv * G, 128), seed=21)
    ks, vs = [], []
    for b, T in enumerate(lens):
        k, v = random_kv(T, Hkv, seed=900 + b)
        ks.append(k)
        vs.append(v)
    _dominant(ks[1], q[1], 15000, 5, G, 400.0)
    _dominant(ks[0], q[0], 12000, 3, G, 30.0)
    c = build_cache(ks, vs, Hkv, merge=False)
    mask = np.zeros((2, Hkv), np.uint8)
    mask[1, 5] = mask[0, 3] = mask[0, 17] = mask[1, 30] = 1
    _decode_check_sampled(c, q, mask, "8-group splits")


@pytest.mark.slow
def test_anchor_decode_sixteen_group_splits_ragged():
    """Splits of 16 groups (four rounds of the rolling fold) over a ragged
    batch of 8 x 16 kv heads, including a one-token sequence and lengths that
    end inside a round; one unit forces the running-maximum path."""
    Hkv, G = 16, 2
    lens = [15000, 3000, 14999, 2049, 8000, 15000, 1, 12345]
    q = random_bf16((len(lens), Hkv * G, 128), seed=22)
    ks, vs = [], []
    for b, T in enumerate(lens):
        k, v = random_kv(T, Hkv, seed=950 + b)
        ks.append(k)
        vs.append(v)
    _dominant(ks[2], q[2], 14000, 7, G, 400.0)
    c = build_cache(ks, vs, Hkv, merge=False)
    mask = np.zeros((len(lens), Hkv), np.uint8)
    for b, h in [(2, 7), (0, 0), (1, 15), (3, 4), (4, 9), (6, 2), (7, 11), (5, 8)]:
        mask[b, h] = 1
    _decode_check_sampled(c, q, mask, "16-group splits")


def gpu_anchor_decode_tail(c, q, kt, vt):
    B, Hq = c.B, q.shape[1]
    out = torch.empty(B, Hq, 128, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, Hq, dtype=torch.float32, device="cuda")
    max_len = max(c.lens)
    ws = lynx.workspace(c.L, B, Hq, 1, max_len)
    note(f"anchor_decode_tail B={B} Hq={Hq} n_tail={0 if kt is None else kt.shape[1]} lens={c.lens[:4]}")
    lynx.lynx_attn_anchor_decode_tail(c.L, B, Hq, max_len, c.lens_dev(), c.table_dev(), c.pool.k_anc,
                                      c.pool.v_anc, c.pool.meta, q.cuda(),
                                      None if kt is None else kt.cuda(),
                                      None if vt is None else vt.cuda(), out, lse, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy()


@pytest.mark.parametrize("n_tail,lens,bt", [(1, [300, 0], None), (8, [1500, 37, 4000], None),
                                            (64, [129, 700], 16), (5, [900, 0, 61], 8)])
def test_anchor_decode_tail(n_tail, lens, bt):
    """Anchor decode that also attends the BF16 tokens generated since the
    context arrived (all n_tail visible); an empty context attends the tail
    alone."""
    Hkv, G = 2, 4
    kv = [random_kv(T, Hkv, seed=1000 + 7 * n_tail + i) for i, T in enumerate(lens)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, bt=bt, seed=n_tail, merge=False)
    B = len(lens)
    q = random_bf16((B, Hkv * G, 128), seed=1100 + n_tail)
    kt = random_bf16((B, n_tail, Hkv, 128), seed=1101 + n_tail)
    vt = random_bf16((B, n_tail, Hkv, 128), seed=1102 + n_tail)
    out, lse = gpu_anchor_decode_tail(c, q, kt, vt)
    ref, ref_lse = oracle.anchor_decode(c.OL, Hkv * G, np.array(c.lens), c.table.numpy(),
                                        c.planes["k_anc"], c.planes["v_anc"], c.meta, bits(q),
                                        k_tail_bits=bits(kt), v_tail_bits=bits(vt))
    assert_close(out, ref, what=f"decode with {n_tail}-token tail")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)


def test_combine_of_more_than_64_splits():
    """One kv head over 40,000 tokens: 79 splits of 512 tokens, merged by the
    combine kernel with its larger load batch (decode with a tail, and
    verification with its causal draft tail)."""
    Hkv, G, T, nq = 1, 4, 40000, 4
    k, v = random_kv(T, Hkv, seed=1300)
    c = build_cache([k], [v], Hkv)
    q = random_bf16((1, Hkv * G, 128), seed=1301)
    kt = random_bf16((1, 8, Hkv, 128), seed=1302)
    vt = random_bf16((1, 8, Hkv, 128), seed=1303)
    out, lse = gpu_anchor_decode_tail(c, q, kt, vt)
    ref, ref_lse = oracle.anchor_decode(c.OL, Hkv * G, np.array(c.lens), c.table.numpy(),
                                        c.planes["k_anc"], c.planes["v_anc"], c.meta, bits(q),
                                        k_tail_bits=bits(kt), v_tail_bits=bits(vt))
    assert_close(out, ref, what="decode with a tail over 79 splits")
    np.testing.assert_allclose(lse, ref_lse, rtol=LSE_RTOL, atol=LSE_ATOL)
    qv = random_bf16((1, nq, Hkv * G, 128), seed=1304)
    kn = random_bf16((1, nq, Hkv, 128), seed=1305)
    vn = random_bf16((1, nq, Hkv, 128), seed=1306)
    got = gpu_verify(c, qv, kn, vn)
    want = oracle_verify(c, qv, kn, vn)
    if isinstance(want, tuple):
        want = want[0]
    assert_close(got, want, what="verification over 79 splits")


def test_anchor_decode_empty_tail_matches_plain_decode():
    Hkv, G = 2, 4
    kv = [random_kv(T, Hkv, seed=1200 + T) for T in (333, 1024)]
    c = build_cache([a for a, _ in kv], [b for _, b in kv], Hkv, merge=False)
    q = random_bf16((2, Hkv * G, 128), seed=1201)
    a, la = gpu_anchor_decode(c, q)
    b, lb = gpu_anchor_decode_tail(c, q, None, None)
    assert np.array_equal(a, b) and np.array_equal(la, lb)


@pytest.mark.parametrize("B,k,V", [(4, 8, 128256), (3, 4, 1001), (37, 1, 12295), (2, 64, 4096)])
def test_spec_accept_greedy(B, k, V):
    """Greedy acceptance, bit-exact against the oracle: random scores with the
    drafts copying the target's choices up to a random point, some positions
    holding a tie between two indices (the lower one wins)."""
    g = torch.Generator().manual_seed(B * 1000 + k + V)
    logits = torch.randn(B, k + 1, V, generator=g)
    choice = logits.argmax(dim=2)
    # plant ties: a second index with the same top score, below or above the first
    for b in range(B):
        for i in range(k + 1):
            if (b + i) % 3 == 0:
                other = int(torch.randint(0, V, (1,), generator=g))
                logits[b, i, other] = logits[b, i, choice[b, i]]
    lg = logits.numpy()
    choice_np = lg.argmax(axis=2)  # first index of the maximum
    drafts = choice_np[:, :k].astype(np.int32).copy()
    cut = torch.randint(0, k + 1, (B,), generator=g).numpy()
    for b in range(B):
        if cut[b] < k:
            drafts[b, cut[b]] = (drafts[b, cut[b]] + 1) % V
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    note(f"spec_accept_greedy B={B} k={k} V={V}")
    lynx.lynx_spec_accept_greedy(torch.from_numpy(lg).cuda(), torch.from_numpy(drafts).cuda(), acc, nxt)
    torch.cuda.synchronize()
    ref_acc, ref_nxt = oracle.accept_greedy(lg, drafts)
    assert np.array_equal(acc.cpu().numpy(), ref_acc)
    assert np.array_equal(nxt.cpu().numpy(), ref_nxt)
    assert np.array_equal(ref_acc, cut)


def _sample_inputs(B, k, V, seed):
    """Target / draft distributions with drafts drawn from q, the uniforms,
    and planted edge cases: drafts outside the vocabulary, p = q rows (no
    residual), all-zero rows, NaN and out-of-range weights, uniforms at 0, 1
    and beyond."""
    rng = np.random.default_rng(seed)
    p = rng.dirichlet(np.full(V, 0.3), size=(B, k + 1)).astype(np.float32)
    q = rng.dirichlet(np.full(V, 0.3), size=(B, k)).astype(np.float32)
    # some draft rows close to the target's, so that drafts are often kept
    mix = rng.random((B, k, 1)).astype(np.float32) < 0.5
    q = np.where(mix, 0.8 * p[:, :k] + 0.2 * q, q).astype(np.float32)
    cq = np.cumsum(q.astype(np.float64), axis=2)
    r = rng.random((B, k, 1)) * cq[:, :, -1:]
    drafts = np.minimum((cq < r).sum(axis=2), V - 1).astype(np.int32)
    u = rng.random((B, k + 1), dtype=np.float32)
    for b in range(B):
        case = b % 8
        if case == 1:
            drafts[b, rng.integers(k)] = V + b        # outside the vocabulary
        elif case == 2:
            drafts[b, 0] = -1
        elif case == 3:
            q[b, 0] = p[b, 0]                        # no residual at a rejection
            u[b, 0] = 1.5
        elif case == 4:
            p[b, 0] = 0.0                            # nothing to draw: -1
            u[b, 0] = 0.9
        elif case == 5:
            p[b, -1, :: max(1, V // 7)] = np.nan     # NaN weights count 0
            p[b, -1, 1::max(1, V // 5)] = 3.0        # above one counts 1
            u[b, :k] = 0.0                           # every draft kept: the bonus
        elif case == 6:
            u[b, k] = 0.0 if b % 16 == 6 else 0.99999994
        elif case == 7:
            u[b, k] = np.nan
    return p, q, drafts, u


@pytest.mark.parametrize("B,k,V", [(8, 8, 128256), (16, 4, 1001), (37, 1, 12295), (9, 64, 4096),
                                   (8, 3, 7), (8, 2, 1), (300, 6, 1000)])
def test_spec_accept_sample(B, k, V):
    """Acceptance of sampled drafts, bit-exact against the oracle (accepted
    counts and drawn tokens) on random distributions and the planted edge
    cases; float4 rows (V % 4 == 0) and scalar rows."""
    p, q, drafts, u = _sample_inputs(B, k, V, seed=B * 7919 + k * 31 + V)
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    nxt = torch.empty(B, dtype=torch.int32, device="cuda")
    note(f"spec_accept_sample B={B} k={k} V={V}")
    lynx.lynx_spec_accept_sample(torch.from_numpy(p).cuda(), torch.from_numpy(q).cuda(),
                                 torch.from_numpy(drafts).cuda(), torch.from_numpy(u).cuda(), acc, nxt)
    torch.cuda.synchronize()
    ref_acc, ref_nxt = oracle.accept_sample(p, q, drafts, u)
    got_acc, got_nxt = acc.cpu().numpy(), nxt.cpu().numpy()
    assert np.array_equal(got_acc, ref_acc), np.nonzero(got_acc != ref_acc)
    assert np.array_equal(got_nxt, ref_nxt), np.nonzero(got_nxt != ref_nxt)
    # the cases cover both outcomes
    assert (ref_acc < k).any() or B < 8
    assert (ref_nxt == -1).any() or B < 5
