"""GPU parity for the adaptation objective (Sec. 3.2): a2t_distill_loss against
the fp64 oracle on the same seeded batches.  Losses within 2e-4 absolute +
1e-4 relative (fp32 statistics over the vocabulary); gradient rows within
1e-4 (fp32 output) or 2^-8 (bf16 output) of each element plus 1e-3 of the
row's largest magnitude; stride padding (filled with NaN) never read into a
result, and written as zeros in the gradient."""
import numpy as np
import pytest

from oracle.distill import KIND_ASR, KIND_NATIVE, distill_losses, row_gradient, row_terms, row_weights
from synth.distill import make_distill_batch

pytestmark = pytest.mark.gpu


def _pad(x, stride, fill):
    out = np.full((x.shape[0], stride), fill, np.float32)
    out[:, :x.shape[1]] = x
    return out


def _run(b, vocab, added, dtype, T, with_grad=True, kind=None):
    import torch
    import paper_2609_31224_amd as a2t
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    ss = (vocab + added + 7) // 8 * 8
    ts = (vocab + 7) // 8 * 8
    s = torch.from_numpy(_pad(b.student, ss, np.nan)).to("cuda").to(tdt)
    t = torch.from_numpy(_pad(b.teacher, ts, np.nan)).to("cuda").to(tdt)
    losses = torch.zeros(5, dtype=torch.float32, device="cuda")
    g = torch.full((b.n, ss), 7.0, dtype=tdt, device="cuda") if with_grad else None
    d = a2t.a2t_distill_create(b.n, vocab, added, a2t.A2T_F32 if dtype == "f32" else a2t.A2T_BF16)
    try:
        a2t.a2t_distill_loss(d, s, t, b.kind if kind is None else kind, b.target, b.dec_group,
                             b.turn_group, T, losses, g)
        torch.cuda.synchronize()
    finally:
        a2t.a2t_distill_destroy(d)
    lo = losses.cpu().numpy().astype(np.float64)
    gr = g.to(torch.float32).cpu().numpy().astype(np.float64) if with_grad else None
    return lo, gr, ss


def _check_losses(lo, ref):
    want = np.array([ref["asr"], ref["native"], ref["dec"], ref["turn"], ref["total"]])
    assert np.all(np.abs(lo - want) <= 2e-4 + 1e-4 * np.abs(want)), (lo, want)


def _check_grad(gr, ref, dtype):
    rel = 1e-4 if dtype == "f32" else 2.0 ** -8
    scale = np.abs(ref).max(axis=1, keepdims=True)
    bad = np.abs(gr - ref) > rel * np.abs(ref) + 1e-3 * scale
    assert not bad.any(), f"{bad.sum()} gradient elements off, first at {np.argwhere(bad)[0]}"


@pytest.mark.parametrize("dtype,T", [("f32", 1.0), ("bf16", 1.0), ("f32", 2.0), ("bf16", 0.5)])
def test_small_batches(gpu, dtype, T):
    vocab, added = 1000, 2
    b = make_distill_batch(seed=11, n_utt=3, units=4, vocab=vocab, added=added, dtype=dtype)
    ref = distill_losses(b.student, b.teacher, b.kind, b.target, b.dec_group, b.turn_group, T)
    lo, gr, ss = _run(b, vocab, added, dtype, T)
    _check_losses(lo, ref.losses)
    _check_grad(gr[:, :vocab + added], ref.grad, dtype)
    assert not gr[:, vocab + added:].any()   # the stride padding of the gradient is zeroed


def test_odd_vocab_masked_rows_and_absent_groups(gpu):
    vocab, added = 997, 2
    b = make_distill_batch(seed=12, n_utt=2, units=5, vocab=vocab, added=added)
    kind = b.kind.copy()
    kind[1::4] = 0                               # rows without loss
    dec = np.where(b.dec_group == 1, -1, b.dec_group).astype(np.int8)  # no "speak" group
    b2 = type(b)(b.student, b.teacher, kind, b.target, dec, b.turn_group)
    ref = distill_losses(b.student, b.teacher, kind, b.target, dec, b.turn_group)
    lo, gr, ss = _run(b2, vocab, added, "f32", 1.0)
    _check_losses(lo, ref.losses)
    _check_grad(gr[:, :vocab + added], ref.grad, "f32")
    assert not gr[kind == 0].any()


def test_loss_only_matches(gpu):
    vocab, added = 1536, 2
    b = make_distill_batch(seed=13, n_utt=2, units=3, vocab=vocab, added=added, dtype="bf16")
    ref = distill_losses(b.student, b.teacher, b.kind, b.target, b.dec_group, b.turn_group)
    lo, _, _ = _run(b, vocab, added, "bf16", 1.0, with_grad=False)
    _check_losses(lo, ref.losses)


def test_full_size_batch(gpu):
    # 16 utterances x 12 units, a vocabulary of 151,936 teacher tokens + 2 added
    vocab, added = 151936, 2
    b = make_distill_batch(seed=14, n_utt=16, units=12, vocab=vocab, added=added, dtype="bf16")
    lo, gr, ss = _run(b, vocab, added, "bf16", 1.0)
    print(f"[distill full] rows {b.n}, GPU losses {lo}", flush=True)
    asr = b.kind == KIND_ASR
    nat = b.kind == KIND_NATIVE
    ce = np.zeros(b.n)
    kl = np.zeros(b.n)
    for r0 in range(0, b.n, 96):                 # oracle rows in chunks (memory)
        sl = slice(r0, r0 + 96)
        ce[sl], kl[sl] = row_terms(b.student[sl], b.teacher[sl], np.where(asr[sl], b.target[sl], -1))
    kl = np.where(nat, kl, 0.0)
    w_ce, w_kl = row_weights(b.kind, b.dec_group, b.turn_group)

    def balanced(groups, G):
        m = [kl[nat & (groups == g)].mean() for g in range(G) if (nat & (groups == g)).any()]
        return float(np.mean(m)) if m else 0.0

    ref = {"asr": ce[asr].mean(), "native": kl[nat].mean(), "dec": balanced(b.dec_group, 3),
           "turn": balanced(b.turn_group, 2)}
    ref["total"] = sum(ref.values())
    _check_losses(lo, ref)
    rows = np.random.default_rng(0).choice(b.n, 24, replace=False)
    want = row_gradient(b.student[rows], b.teacher[rows], np.where(asr[rows], b.target[rows], -1),
                        w_ce[rows], w_kl[rows])
    _check_grad(gr[rows, :vocab + added], want, "bf16")


def test_argument_errors(gpu):
    import torch
    import paper_2609_31224_amd as a2t
    lib = a2t.raw_lib()
    import ctypes as C
    d = a2t.a2t_distill_create(8, 64, 2, a2t.A2T_F32)
    try:
        s = torch.zeros(4, 72, device="cuda")
        t = torch.zeros(4, 64, device="cuda")
        losses = torch.zeros(5, device="cuda")
        kind = np.array([1, 2, 2, 0], np.int8)
        tgt = np.array([3, -1, -1, -1], np.int32)
        dec = np.array([-1, 0, -1, -1], np.int8)
        turn = np.array([-1, -1, 1, -1], np.int8)
        P8, P32 = C.POINTER(C.c_int8), C.POINTER(C.c_int32)

        def call(n=4, ss=72, ts=64, k=kind, tg=tgt, T=1.0, sp=s.data_ptr()):
            return lib.a2t_distill_loss(d.ptr, n, sp, ss, t.data_ptr(), ts, k.ctypes.data_as(P8),
                                        tg.ctypes.data_as(P32), dec.ctypes.data_as(P8),
                                        turn.ctypes.data_as(P8), T, losses.data_ptr(), None)
        assert call() == a2t.A2T_OK
        assert call(n=9) == a2t.A2T_ERR_INVALID          # beyond max_rows
        assert call(ss=70) == a2t.A2T_ERR_INVALID        # stride not a multiple of 8
        assert call(ss=64) == a2t.A2T_ERR_INVALID        # stride below vocab + added
        assert call(sp=s.data_ptr() + 4) == a2t.A2T_ERR_INVALID  # misaligned
        assert call(T=0.0) == a2t.A2T_ERR_INVALID
        assert call(k=np.array([1, 2, 3, 0], np.int8)) == a2t.A2T_ERR_INVALID
        assert call(tg=np.array([66, -1, -1, -1], np.int32)) == a2t.A2T_ERR_INVALID
        assert call() == a2t.A2T_OK                       # still usable
        torch.cuda.synchronize()
    finally:
        a2t.a2t_distill_destroy(d)
