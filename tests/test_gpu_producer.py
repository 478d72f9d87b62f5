"""GPU parity of the fused K/V producer (tm_qkv_produce) against the oracle.

The producer RMS-normalises every (token, head) row of the chunk's queries and
keys (oracle: ``oracle.rms_normalise`` in fp64) and appends the normalised keys
and the values to the cache. Checks:
- q_out and the cached K rows: a bf16 result must be one of the two bf16
  neighbours of the exact (fp64) value, since the kernel computes in fp32
  (relative error ~1e-6) and rounds once; an fp32 result must agree to 1e-5
  relative;
- the V pool and the cache bookkeeping: bit for bit equal to what
  tm_kv_append produces from the same chunk (the values are copied);
- attention on the produced cache equals the oracle's attention on the
  oracle-normalised inputs, to the usual bar;
- a full-size 480p chunk on sampled heads and rows.
Inputs are seeded normal draws with a different scale per row, so that the
normalisation has work to do.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import assert_close, assert_rounds_to, say
from oracle import ChunkGeometry, StreamHistory, rms_normalise
from synth import bf16_bits_to_f32, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tm():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2506_03099_amd import tm as binding
    binding.lib()
    return binding


def _raw(rng, shape, dtype, scaled=True):
    """Seeded raw activations [B, n, H, D]: normal draws times a per-row scale
    in [0.05, 20]; returns (device tensor, exact fp32 values)."""
    x = rng.standard_normal(shape).astype(np.float32)
    if scaled:
        x *= np.exp(rng.uniform(np.log(0.05), np.log(20.0), size=shape[:-1] + (1,))).astype(np.float32)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        vals = bf16_bits_to_f32(bits)
        t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()
        return t, vals
    return torch.from_numpy(x).cuda(), x


def _assert_normalised(got, want64, dtype, what):
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == want64.shape, (got.shape, want64.shape)
    assert np.all(np.isfinite(got)), what
    if dtype == "bf16":
        # ulp of bf16 at |want|: 2^(floor(log2|want|) - 7)
        mag = np.abs(want64)
        ulp = np.where(mag > 0, 2.0 ** (np.floor(np.log2(np.maximum(mag, 1e-300))) - 7), 0.0)
        bad = np.abs(got - want64) > ulp
    else:
        bad = np.abs(got - want64) > 1e-5 * np.abs(want64) + 1e-30
    assert not bad.any(), f"{what}: {int(bad.sum())} elements off, e.g. got {got[bad][:3]} want {want64[bad][:3]}"


def _k_rows(cache, chunk, B, H, D):
    """Cached K rows of `chunk` as fp32 [B, n, H, D]."""
    off, n = cache.locate(chunk)
    k = cache.k_pool[:, :, off:off + n, :].float().cpu().numpy()
    return k.transpose(0, 2, 1, 3)


def _gain(rng, H, D):
    return torch.from_numpy(rng.uniform(0.5, 2.0, size=(H, D)).astype(np.float32)).cuda()


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("bf16", 64), ("f32", 128), ("f32", 64)])
def test_producer_matches_oracle_and_append(tm, dtype, D):
    B, H, T, C, R, W = 2, 3, 5, 2, 2, 1
    say(f"qkv_produce vs oracle: dtype={dtype} D={D}")
    rng = np.random.default_rng(1000 + D + (dtype == "bf16"))
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype)
    prod, ref = tm.KVCache(desc), tm.KVCache(desc)
    for c in (prod, ref):  # same canary bits in both pools
        c.k_pool.view(torch.uint8).fill_(0x5A)
        c.v_pool.view(torch.uint8).fill_(0x3C)
    qg, kg = _gain(rng, H, D), _gain(rng, H, D)
    gains = dict(q_gain=qg, k_gain=kg, eps=1e-3)
    qg_h, kg_h = qg.cpu().numpy(), kg.cpu().numpy()
    written = np.zeros(prod.capacity, bool)
    # c_0, then chunks of full and ragged lengths, one overwrite of the latest
    # chunk, and enough chunks to evict through the ring
    for chunk, n, use_gain in [(0, R * T, True), (1, C * T, False), (2, 7, True), (2, 3, True),
                               (3, C * T, False), (4, 1, True)]:
        q, qv = _raw(rng, (B, n, H, D), dtype)
        k, kv = _raw(rng, (B, n, H, D), dtype)
        v, _ = _raw(rng, (B, n, H, D), dtype)
        kw = gains if use_gain else {}
        q_out = tm.tm_qkv_produce(prod, chunk, q, k, v, **kw)
        tm.tm_kv_append(ref, chunk, k, v)
        torch.cuda.synchronize()
        g_q = qg_h if use_gain else None
        g_k = kg_h if use_gain else None
        eps = 1e-3 if use_gain else 0.0
        _assert_normalised(q_out.float().cpu().numpy(), rms_normalise(qv, g_q, eps), dtype,
                           f"q_out chunk {chunk}")
        _assert_normalised(_k_rows(prod, chunk, B, H, D), rms_normalise(kv, g_k, eps), dtype,
                           f"cached K chunk {chunk}")
        # V pool and bookkeeping: as tm_kv_append; K rows never written keep
        # the canary
        assert torch.equal(prod.v_pool.view(torch.uint8), ref.v_pool.view(torch.uint8)), chunk
        assert prod.latest() == ref.latest() == chunk
        assert prod.locate(chunk) == ref.locate(chunk)
        off, nn = prod.locate(chunk)
        written[off:off + nn] = True
        untouched = prod.k_pool.view(torch.uint8)[:, :, torch.from_numpy(~written).cuda()]
        assert bool((untouched == 0x5A).all()), chunk


def test_producer_in_place_and_errors(tm):
    B, H, D, T, C, R, W = 1, 2, 128, 8, 2, 1, 1
    say("qkv_produce in place and argument errors")
    rng = np.random.default_rng(7)
    desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
    cache = tm.KVCache(desc)
    q, qv = _raw(rng, (B, R * T, H, D), "bf16")
    k, _ = _raw(rng, (B, R * T, H, D), "bf16")
    v, _ = _raw(rng, (B, R * T, H, D), "bf16")
    out = tm.tm_qkv_produce(cache, 0, q, k, v, q_out=q)  # in place
    assert out is q
    torch.cuda.synchronize()
    _assert_normalised(q.float().cpu().numpy(), rms_normalise(qv), "bf16", "in-place q")
    q2, _ = _raw(rng, (B, C * T, H, D), "bf16")
    k2, _ = _raw(rng, (B, C * T, H, D), "bf16")
    v2, _ = _raw(rng, (B, C * T, H, D), "bf16")
    for kw in [dict(eps=-1.0), dict(eps=float("nan")), dict(q_out=k2)]:
        with pytest.raises(tm.TMError) as e:
            tm.tm_qkv_produce(cache, 1, q2, k2, v2, **kw)
        assert e.value.status == tm.TM_E_ARG
        assert cache.latest() == 0  # nothing was appended
    with pytest.raises(tm.TMError) as e:  # out of order
        tm.tm_qkv_produce(cache, 2, q2, k2, v2)
    assert e.value.status == tm.TM_E_ORDER
    with pytest.raises(tm.TMError) as e:  # more tokens than a chunk holds
        big, _ = _raw(rng, (B, C * T + 1, H, D), "bf16")
        tm.tm_qkv_produce(cache, 1, big, big, big)
    assert e.value.status == tm.TM_E_CAPACITY


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_producer_then_attention_matches_oracle(tm, dtype):
    # raw q, k, v -> producer -> attention, against the oracle's attention on
    # the oracle-normalised (and, for bf16, rounded) queries and keys
    B, H, D, T, C, R, W = 1, 2, 128, 50, 3, 3, 1
    say(f"qkv_produce + attention: dtype={dtype}")
    rng = np.random.default_rng(11)
    desc = tm.make_desc(B, H, D, T, C, R, W, dtype)
    cache = tm.KVCache(desc)
    g = ChunkGeometry(T, C, R, W)
    hist = StreamHistory(g)

    def exact(x64):
        x32 = x64.astype(np.float32)
        return bf16_bits_to_f32(f32_to_bf16_bits(x32)) if dtype == "bf16" else x32

    for chunk in range(4):
        n = R * T if chunk == 0 else C * T
        q, qv = _raw(rng, (B, n, H, D), dtype)
        k, kv = _raw(rng, (B, n, H, D), dtype)
        v, vv = _raw(rng, (B, n, H, D), dtype, scaled=False)
        qn = tm.tm_qkv_produce(cache, chunk, q, k, v)
        o = tm.tm_sparse_causal_attn_fwd(desc, qn, chunk, cache=cache)
        hist.append(chunk, exact(rms_normalise(kv)), vv)
        want, _ = hist.attend(exact(rms_normalise(qv)), chunk)
        if dtype == "bf16":  # the arithmetic through the fp32 output; bf16 = its rounding
            of = tm.tm_sparse_causal_attn_fwd_f32out(desc, qn, chunk, cache=cache)
            torch.cuda.synchronize()
            assert_rounds_to(o, of, f"chunk {chunk}")
            o = of
        torch.cuda.synchronize()
        assert_close(o.float().cpu().numpy(), want, dtype, f"chunk {chunk}")


def test_producer_480p_chunk_sampled(tm):
    # the WAN-14B 480p chunk: 4680 tokens x 40 heads x 128, bf16
    B, H, D, T, C, R, W = 1, 40, 128, 1560, 3, 1, 1
    say("qkv_produce 480p chunk, sampled")
    rng = np.random.default_rng(480)
    desc = tm.make_desc(B, H, D, T, C, R, W, "bf16")
    prod, ref = tm.KVCache(desc), tm.KVCache(desc)
    for c in (prod, ref):  # same canary bits in the rows neither call writes
        c.v_pool.view(torch.uint8).fill_(0x3C)
    qg, kg = _gain(rng, H, D), _gain(rng, H, D)
    for chunk, n in [(0, R * T), (1, C * T)]:
        q, qv = _raw(rng, (B, n, H, D), "bf16")
        k, kv = _raw(rng, (B, n, H, D), "bf16")
        v, _ = _raw(rng, (B, n, H, D), "bf16")
        q_out = tm.tm_qkv_produce(prod, chunk, q, k, v, q_gain=qg, k_gain=kg, eps=1e-6)
        tm.tm_kv_append(ref, chunk, k, v)
        torch.cuda.synchronize()
        rows = np.sort(rng.choice(n, size=min(n, 257), replace=False))
        heads = [0, 17, 39]
        qo = q_out[:, rows][:, :, heads].float().cpu().numpy()
        want_q = rms_normalise(qv[:, rows][:, :, heads], qg.cpu().numpy()[heads], 1e-6)
        _assert_normalised(qo, want_q, "bf16", f"q_out chunk {chunk}")
        off, nn = prod.locate(chunk)
        kk = prod.k_pool[:, heads][:, :, off + rows].float().cpu().numpy().transpose(0, 2, 1, 3)
        want_k = rms_normalise(kv[:, rows][:, :, heads], kg.cpu().numpy()[heads], 1e-6)
        _assert_normalised(kk, want_k, "bf16", f"cached K chunk {chunk}")
        assert torch.equal(prod.v_pool.view(torch.uint8), ref.v_pool.view(torch.uint8))
