"""GPU parity of the serializer / deserializer (Sec. 4.2, Sec. 5) through the
C ABI, bit for bit against the CPU oracle on the same seeded inputs: the
transmission buffers of objects (ragged lengths, several kv heads, outlier
and adversarial values), their scatter into a paged pool delivered in
shuffled order, the residual phase into code planes, and a full 32K-token
Llama-3-8B layer as one object."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx
from tests.gpu_cases import bits, note, random_kv

pytestmark = pytest.mark.gpu


def gpu_serialize(Hkv, n, k, v):
    na, nr = lynx.lynx_serialized_bytes(Hkv, n)
    anc = torch.full((na,), 0xA5, dtype=torch.uint8, device="cuda")
    res = torch.full((nr,), 0xA5, dtype=torch.uint8, device="cuda")
    note(f"serialize Hkv={Hkv} n={n}")
    lynx.lynx_kv_serialize(Hkv, n, k.cuda(), v.cuda(), anc, res)
    torch.cuda.synchronize()
    return anc, res


@pytest.mark.parametrize("n,Hkv", [(1, 1), (16, 2), (127, 1), (128, 4), (129, 2), (700, 3),
                                   (2048, 8)])
def test_serialize_bit_exact(n, Hkv):
    k, v = random_kv(n, Hkv, seed=500 + n + Hkv)
    anc, res = gpu_serialize(Hkv, n, k, v)
    ra, rr = oracle.serialize(Hkv, n, bits(k), bits(v))
    assert np.array_equal(anc.cpu().numpy(), ra), f"anchor buffer: {np.count_nonzero(anc.cpu().numpy() != ra)} bytes differ"
    assert np.array_equal(res.cpu().numpy(), rr)


def test_serialize_adversarial_values():
    """Constant and two-valued groups, signed zeros, denormals, huge values and
    rounding ties in an object whose last K group is ragged."""
    n, Hkv = 260, 2
    g = torch.Generator().manual_seed(7)
    x = torch.randn(n, Hkv, 128, generator=g)
    x[:, 0, 0] = 3.25
    x[:, 0, 1] = torch.where(torch.arange(n) % 3 == 0, -7.0, 9.0)
    x[:, 0, 2] = -0.0
    x[:, 0, 3] = torch.randn(n, generator=g) * 1e-39
    x[:, 1, 4] = torch.randn(n, generator=g) * 1e37
    x[:, 1, 5] = torch.arange(n) % 256
    v = torch.randn(n, Hkv, 128, generator=g)
    v[0] = 1.5
    v[2, :, :4] = torch.tensor([0.0, 255.0, 126.5, 2.5])
    v[2, :, 4:] = 0.0
    k, v = x.to(torch.bfloat16), v.to(torch.bfloat16)
    anc, res = gpu_serialize(Hkv, n, k, v)
    ra, rr = oracle.serialize(Hkv, n, bits(k), bits(v))
    assert np.array_equal(anc.cpu().numpy(), ra)
    assert np.array_equal(res.cpu().numpy(), rr)


@pytest.mark.parametrize("T,cuts,bt", [(700, [0, 256, 640], 16), (1000, [0, 512], 32),
                                       (129, [0, 128], 8), (4096, [0, 1024, 2048, 3072], 16)])
def test_deserialize_into_paged_pool(T, cuts, bt):
    """Objects serialized on the GPU, delivered in reverse order into a paged
    pool (random block table): anchor phase, then residual phase; pool planes,
    metadata and codes against the oracle's deserializer."""
    Hkv = 2
    k, v = random_kv(T, Hkv, seed=900 + T)
    max_tokens = T + 50
    nb = -(-max_tokens // bt)
    n_blocks = nb + 5
    table = torch.randperm(n_blocks, generator=torch.Generator().manual_seed(T))[:nb].to(torch.int32).view(1, -1)
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt, max_blocks_per_seq=nb, num_blocks=n_blocks,
                    max_tokens=max_tokens)
    OL = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=nb, max_tokens=max_tokens)
    pool = lynx.KVPool.allocate(L, 1)
    tdev = table.cuda()
    bounds = list(cuts) + [T]
    objs = [(bounds[i], bounds[i + 1] - bounds[i]) for i in range(len(cuts))]
    bufs = {t0: gpu_serialize(Hkv, n, k[t0:t0 + n], v[t0:t0 + n]) for t0, n in objs}
    for t0, n in reversed(objs):
        note(f"deserialize_anchor t0={t0} n={n} bt={bt}")
        lynx.lynx_kv_deserialize_anchor(L, 0, t0, n, tdev, bufs[t0][0], pool.k_anc, pool.v_anc, pool.meta)
    for t0, n in objs:
        note(f"deserialize_residual t0={t0} n={n} bt={bt}")
        lynx.lynx_kv_deserialize_residual(L, 0, t0, n, tdev, bufs[t0][1], pool.k_anc, pool.v_anc,
                                          pool.k_codes, pool.v_codes)
    torch.cuda.synchronize()
    nbytes = oracle.plane_bytes(OL, n_blocks, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    meta = oracle.Meta.empty(OL, 1)
    codes = {name: np.zeros(2 * nbytes, np.uint8) for name in ("k_codes", "v_codes")}
    for t0, n in objs:
        ra, rr = oracle.serialize(Hkv, n, bits(k[t0:t0 + n]), bits(v[t0:t0 + n]))
        oracle.deserialize_anchor(OL, 0, t0, n, table.numpy(), ra, planes, meta)
        oracle.deserialize_residual(OL, 0, t0, n, table.numpy(), rr, planes, codes)
    for name in ("k_anc", "v_anc"):
        assert np.array_equal(getattr(pool, name).cpu().numpy(), planes[name]), name
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        got = getattr(pool.meta, name).cpu().numpy()
        assert np.array_equal(got.view(np.uint32), getattr(meta, name).view(np.uint32)), name
    for name in ("k_codes", "v_codes"):
        assert np.array_equal(getattr(pool, name).cpu().numpy(), codes[name]), name


def test_llama3_8b_layer_as_one_object():
    """A full 32K-token, 8-kv-head layer of the Llama-3-8B workload serialized
    as one object: buffers bit-exact against the oracle, and scattered into a
    contiguous pool they equal the sequence encode of the same layer."""
    w = inputs.WORKLOADS["llama3-8b-32k"]
    T, Hkv = w.context, w.Hkv
    k = inputs.kv(w, "k", layer=3)
    v = inputs.kv(w, "v", layer=3)
    anc, res = gpu_serialize(Hkv, T, k, v)
    ra, rr = oracle.serialize(Hkv, T, bits(k), bits(v))
    assert np.array_equal(anc.cpu().numpy(), ra)
    assert np.array_equal(res.cpu().numpy(), rr)
    L = lynx.contiguous_layout(Hkv, 1, T)
    table = torch.zeros(1, 1, dtype=torch.int32, device="cuda")
    direct = lynx.KVPool.allocate(L, 1)
    note("encode 32K layer")
    direct.encode(0, T, table, k.cuda(), v.cuda())
    direct.merge()
    recv = lynx.KVPool.allocate(L, 1)
    note("deserialize 32K layer")
    lynx.lynx_kv_deserialize_anchor(L, 0, 0, T, table, anc, recv.k_anc, recv.v_anc, recv.meta)
    lynx.lynx_kv_deserialize_residual(L, 0, 0, T, table, res, recv.k_anc, recv.v_anc, recv.k_codes,
                                      recv.v_codes)
    torch.cuda.synchronize()
    for name in ("k_anc", "v_anc", "k_codes", "v_codes"):
        assert torch.equal(getattr(recv, name), getattr(direct, name)), name
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        assert torch.equal(getattr(recv.meta, name), getattr(direct.meta, name)), name
