"""GPU parity of the audio cross-attention (tm_audio_cross_attn_fwd) against
the oracle (``oracle.audio_cross_attention``, fp32 on the same bf16 values).

Every call runs twice, with the bf16 output and with the fp32 output of the
same kernel (tm_audio_cross_attn_fwd_f32out). Face rows of the fp32 output are
compared element by element with the bf16 bar, max |err| <= 2e-2 x RMS over
the compared rows, and the bf16 output must be the nearest-even rounding of the
fp32 output, bit for bit. (A window holds at most a few hundred keys, 160 in
the paper's setting, so |o| reaches several times its RMS and the rounding of
the bf16 format alone comes close to the bar.) Rows without a face, and rows
whose face id is outside [0, M), must be exactly zero in both outputs. Cases: ragged row blocks and a partial last frame, windows clipped at
both ends of the audio, a window padded to the next 32 keys, several streams
mixed inside one 32-row block, frames split over several workgroups, the
largest window that fits in LDS, in-place output, no rows, rows that use no
stream 0, more dense face blocks than compute waves (with the queries staged in
LDS and, for windows too long for that, gathered into registers), more rows
than one zero-fill workgroup stages at once, and the 480p
workloads (two faces in full, one face on sampled heads and rows).
"""
import numpy as np
import pytest
import torch

from gpu_helpers import assert_close, assert_rounds_to, say
from oracle import audio_cross_attention
from synth import AUDIO_WORKLOADS, bf16_bits_to_f32, draw_audio, f32_to_bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tm():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2506_03099_amd import tm as binding
    binding.lib()
    return binding


def _bf16(rng, shape, norm):
    x = rng.standard_normal(shape).astype(np.float32)
    if norm:
        x /= np.sqrt(np.mean(x * x, axis=-1, keepdims=True))
    bits = f32_to_bf16_bits(x)
    return bf16_bits_to_f32(bits), bits


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _inputs(seed, B, n, H, D, M, La):
    rng = np.random.default_rng(seed)
    q, qb = _bf16(rng, (B, n, H, D), True)
    ak, akb = _bf16(rng, (B, M, La, H, D), True)
    av, avb = _bf16(rng, (B, M, La, H, D), False)
    return rng, (q, ak, av), (_dev(qb), _dev(akb), _dev(avb))


def _run(tm, desc, qd, first, akd, avd, faced, **kw):
    """(bf16 output, fp32 output) of the same call."""
    o = tm.tm_audio_cross_attn_fwd(desc, qd, first, akd, avd, faced, **kw)
    kw.pop("o", None)
    of = tm.tm_audio_cross_attn_fwd_f32out(desc, qd, first, akd, avd, faced, **kw)
    torch.cuda.synchronize()
    return o, of


def _check(o_pair, q, ak, av, face, T, A, first, w, what, heads=None, rows=None):
    o_dev, of_dev = o_pair
    assert_rounds_to(o_dev, of_dev, what)
    M = ak.shape[1]
    valid = np.where((face >= 0) & (face < M), face, -1)  # other ids mean no face
    o = of_dev.cpu().numpy()
    if heads is not None:
        o = o[:, :, heads]
    if rows is not None:
        o = o[:, rows]
        valid_r = valid[:, rows]
    else:
        valid_r = valid
    want = audio_cross_attention(q, ak, av, valid, tokens_per_frame=T, audio_per_frame=A,
                                 first_frame=first, half_window=w, heads=heads, rows=rows)
    sel = valid_r >= 0
    assert np.all(o[~sel] == 0), f"{what}: rows without a face are not zero"
    assert sel.any()
    assert_close(o[sel], want[sel], "bf16", what)


@pytest.mark.parametrize("D", [128, 64])
@pytest.mark.parametrize("first", [0, 2, 6])
def test_audio_matches_oracle_small(tm, D, first):
    B, H, T, A, Fa, M, w, frames = 2, 3, 50, 7, 9, 3, 2, 3
    say(f"audio vs oracle: D={D} first_frame={first}")
    n = T * frames
    rng, (q, ak, av), (qd, akd, avd) = _inputs(100 + D + first, B, n, H, D, M, Fa * A)
    face = rng.choice([-1, 0, 1, 2, 3, 7, -5], size=(B, n),
                      p=[0.25, 0.2, 0.2, 0.2, 0.05, 0.05, 0.05]).astype(np.int32)
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, first, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, first, w, f"D={D} first={first}")


@pytest.mark.parametrize("D", [128, 64])
def test_audio_stream_zero_unused_and_many_face_blocks(tm, D):
    """Rows of streams 1 and 2 only (the kernel's window loads for stream 0,
    issued before the face ids are known, are dropped), and a frame whose rows
    are nearly all faces (more dense 32-row blocks than compute waves)."""
    B, H, T, A, Fa, M, w, frames = 1, 2, 700, 16, 8, 3, 2, 3
    say(f"audio without stream 0: D={D}")
    n = T * frames
    rng, (q, ak, av), (qd, akd, avd) = _inputs(300 + D, B, n, H, D, M, Fa * A)
    face = rng.choice([-1, 1, 2], size=(B, n), p=[0.3, 0.35, 0.35]).astype(np.int32)
    face[:, T:2 * T] = np.where(rng.random((B, T)) < 0.95, 2, -1)  # frame 1: one stream, 95% of rows
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, 1, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, 1, w, f"no stream 0 D={D}")


@pytest.mark.parametrize("D,A", [(128, 40), (64, 100)])
def test_audio_unstaged_queries_many_streams_and_blocks(tm, D, A):
    """Windows too long for the per-wave query slots beside them in LDS
    (200 keys at D = 128, 500 at D = 64): queries gathered into registers and
    outputs stored from them, with three streams, rows of stream 0 missing in
    one frame and a frame whose rows are nearly all one face (more dense blocks
    than waves, so waves gather a second block)."""
    B, H, T, Fa, M, w, frames = 1, 2, 700, 8, 3, 2, 3
    say(f"audio unstaged: D={D} keys={5 * A}")
    n = T * frames
    rng, (q, ak, av), (qd, akd, avd) = _inputs(600 + D, B, n, H, D, M, Fa * A)
    face = rng.choice([-1, 0, 1, 2], size=(B, n), p=[0.25, 0.25, 0.25, 0.25]).astype(np.int32)
    face[:, T:2 * T] = np.where(rng.random((B, T)) < 0.95, 1, -1)
    face[:, 2 * T:] = np.where(face[:, 2 * T:] == 0, 2, face[:, 2 * T:])
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, 2, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, 2, w, f"unstaged D={D}")


@pytest.mark.parametrize("T,A,n_extra", [(70, 32, 35), (1100, 33, 100), (2100, 32, 0), (4200, 32, 50)])
def test_audio_ragged_rows_split_frames_and_padded_windows(tm, T, A, n_extra):
    # T = 70: blocks of 32, 32, 6 rows; T = 1100: 35 blocks, one workgroup per
    # frame; T = 2100: 66 blocks, two workgroups per frame taking every other
    # block; T = 4200: 132 blocks, three workgroups; A = 33: 165 keys padded to
    # 192; a partial last frame
    B, H, D, Fa, M, w, first = 1, 2, 128, 6, 2, 2, 1
    n = 2 * T + n_extra
    say(f"audio ragged: T={T} A={A} n={n}")
    rng, (q, ak, av), (qd, akd, avd) = _inputs(T + A, B, n, H, D, M, Fa * A)
    face = rng.choice([-1, 0, 1], size=(B, n)).astype(np.int32)
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, first, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, first, w, f"T={T} A={A}")


@pytest.mark.parametrize("w,Fa,A", [(0, 5, 16), (1, 5, 16), (10, 4, 16)])
def test_audio_window_extremes(tm, w, Fa, A):
    # w = 0: a frame's own audio only; w = 10 over 4 frames: all audio
    B, H, D, T, M = 1, 2, 128, 40, 1
    frames = min(Fa, 3)
    n = T * frames
    say(f"audio window w={w} Fa={Fa}")
    rng, (q, ak, av), (qd, akd, avd) = _inputs(7 + w, B, n, H, D, M, Fa * A)
    face = np.where(rng.random((B, n)) < 0.7, 0, -1).astype(np.int32)
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, 0, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, 0, w, f"w={w}")


@pytest.mark.parametrize("D,A", [(128, 57), (64, 121)])
def test_audio_largest_window_that_fits(tm, D, A):
    # (2w + 1) * A = 285 keys padded to 288 at D = 128, 605 padded to 608 at
    # D = 64: the LDS limit
    B, H, T, Fa, M, w = 1, 2, 64, 5, 1, 2
    n = T
    say(f"audio largest window: D={D} A={A}")
    rng, (q, ak, av), (qd, akd, avd) = _inputs(D + A, B, n, H, D, M, Fa * A)
    face = np.zeros((B, n), dtype=np.int32)
    face[:, ::5] = -1
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, 2, akd, avd, torch.from_numpy(face).cuda())
    _check(o, q, ak, av, face, T, A, 2, w, f"D={D} keys={5 * A}")
    with pytest.raises(tm.TMError) as e:  # one more key per frame no longer fits
        tm.tm_audio_cross_attn_fwd(tm.make_audio_desc(B, H, D, T, A + 1, Fa, M, w), qd, 2,
                                   akd, avd, torch.from_numpy(face).cuda())
    assert e.value.status == tm.TM_E_SHAPE


def test_audio_in_place_deterministic_and_empty(tm):
    B, H, D, T, A, Fa, M, w = 1, 4, 128, 96, 32, 7, 2, 2
    n = 3 * T
    say("audio in place, determinism, no rows")
    rng, (q, ak, av), (qd, akd, avd) = _inputs(55, B, n, H, D, M, Fa * A)
    face_np = rng.choice([-1, 0, 1], size=(B, n)).astype(np.int32)
    face = torch.from_numpy(face_np).cuda()
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o1 = _run(tm, desc, qd, 3, akd, avd, face)
    o2 = tm.tm_audio_cross_attn_fwd(desc, qd, 3, akd, avd, face)
    qq = qd.clone()
    o3 = tm.tm_audio_cross_attn_fwd(desc, qq, 3, akd, avd, face, o=qq)
    torch.cuda.synchronize()
    assert o3 is qq
    assert torch.equal(o1[0].view(torch.int16), o2.view(torch.int16))
    assert torch.equal(o1[0].view(torch.int16), qq.view(torch.int16))
    # an fp32 output may not start at (or overlap) the bf16 queries: q is a
    # bf16 view of the first half of the fp32 buffer given as o
    buf = torch.empty(qd.shape, dtype=torch.float32, device="cuda")
    q_alias = buf.view(torch.bfloat16).view(-1)[:qd.numel()].view(qd.shape)
    q_alias.copy_(qd)
    with pytest.raises(tm.TMError) as e:
        tm.tm_audio_cross_attn_fwd_f32out(desc, q_alias, 3, akd, avd, face, o=buf)
    assert e.value.status == tm.TM_E_ARG
    _check(o1, q, ak, av, face_np, T, A, 3, w, "in place")
    canary = torch.full_like(qd, 3.0)
    tm.tm_audio_cross_attn_fwd(desc, qd, 3, akd, avd, face, o=canary, n_tok=0)
    torch.cuda.synchronize()
    assert bool((canary == 3.0).all())


def test_audio_480p_two_faces_full(tm):
    w = AUDIO_WORKLOADS["wan14b_480p_audio_2faces"]
    say(f"audio {w.name}: {w.n_tok} rows x {w.heads} heads, frames {w.first_frame}.., two faces")
    d = draw_audio(w)
    desc = tm.make_audio_desc(w.batch, w.heads, w.head_dim, w.tokens_per_frame, w.audio_per_frame,
                              w.audio_frames, w.streams, w.half_window)
    o = _run(tm, desc, _dev(d["q_bits"]), w.first_frame, _dev(d["ak_bits"]), _dev(d["av_bits"]),
             torch.from_numpy(d["face"]).cuda())
    _check(o, d["q"], d["ak"], d["av"], d["face"], w.tokens_per_frame, w.audio_per_frame,
           w.first_frame, w.half_window, w.name)


def test_audio_many_rows_zero_fill_in_batches(tm):
    """More compute workgroups than CUs (8 heads x 40 frames) and 40000 rows:
    each zero-fill workgroup covers more rows than one batch of face flags
    (512), so it stages several batches. Every row without a face must be
    zero in all heads; face rows are compared on a sample."""
    B, H, D, T, A, M, w, frames = 1, 8, 64, 1000, 16, 2, 2, 40
    n = T * frames
    Fa = frames + 2
    say(f"audio many rows: n={n}, {H} heads")
    rng, (q, ak, av), (qd, akd, avd) = _inputs(77, B, n, H, D, M, Fa * A)
    face = rng.choice([-1, 0, 1, 5], size=(B, n), p=[0.55, 0.2, 0.2, 0.05]).astype(np.int32)
    desc = tm.make_audio_desc(B, H, D, T, A, Fa, M, w)
    o = _run(tm, desc, qd, 1, akd, avd, torch.from_numpy(face).cuda())
    on = torch.from_numpy((face >= 0) & (face < M)).cuda()
    assert bool((o[0][~on] == 0).all()) and bool((o[1][~on] == 0).all()), "rows without a face are not zero"
    rows = np.sort(rng.choice(n, 400, replace=False))
    _check(o, q, ak, av, face, T, A, 1, w, "many rows", heads=[0, 5, 7], rows=rows)


def test_audio_480p_chunk_sampled(tm):
    w = AUDIO_WORKLOADS["wan14b_480p_audio_chunk"]
    say(f"audio {w.name}: {w.n_tok} rows x {w.heads} heads, sampled")
    d = draw_audio(w)
    desc = tm.make_audio_desc(w.batch, w.heads, w.head_dim, w.tokens_per_frame, w.audio_per_frame,
                              w.audio_frames, w.streams, w.half_window)
    o = _run(tm, desc, _dev(d["q_bits"]), w.first_frame, _dev(d["ak_bits"]), _dev(d["av_bits"]),
             torch.from_numpy(d["face"]).cuda())
    # every row without a face is zero (all heads); face rows sampled
    on = torch.from_numpy(d["face"] >= 0).cuda()
    assert bool((o[0][~on] == 0).all()) and bool((o[1][~on] == 0).all())
    rng = np.random.default_rng(3)
    face_rows = np.flatnonzero(d["face"][0] >= 0)
    rows = np.sort(np.concatenate([rng.choice(face_rows, 160, replace=False),
                                   rng.choice(np.flatnonzero(d["face"][0] < 0), 32, replace=False)]))
    _check(o, d["q"], d["ak"], d["av"], d["face"], w.tokens_per_frame, w.audio_per_frame,
           w.first_frame, w.half_window, w.name, heads=[0, 13, 39], rows=rows)
