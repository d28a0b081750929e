"""Pins for the oracle of the adaptation objective (Sec. 3.2): masked CE over
transcription rows, T^2 KL(P_T || P_S) at native rows with the teacher extended
by zero probability on the added tokens, group-balanced means, and the
gradient with respect to the student logits."""
import numpy as np
import pytest
import torch

from oracle.distill import KIND_ASR, KIND_NATIVE, distill_losses, row_weights
from synth.distill import make_distill_batch


def _torch_reference(b, T):
    # an independent computation with torch float64 on the CPU: kl_div,
    # cross_entropy and autograd for the gradient
    s = torch.tensor(b.student, dtype=torch.float64, requires_grad=True)
    t = torch.tensor(b.teacher, dtype=torch.float64)
    V = t.shape[1]
    kind = torch.tensor(b.kind.astype(np.int64))
    nat = kind == KIND_NATIVE
    asr = kind == KIND_ASR
    logp_s = torch.log_softmax(s / T, dim=1)
    logp_t = torch.log_softmax(t / T, dim=1)
    # teacher zero on the added tokens: only the first V student log-probs enter
    kl = T * T * torch.nn.functional.kl_div(logp_s[:, :V], logp_t, reduction="none",
                                            log_target=True).sum(dim=1)
    ce = torch.nn.functional.cross_entropy(s[asr], torch.tensor(b.target[b.kind == KIND_ASR],
                                                                dtype=torch.int64), reduction="none")
    terms = [ce.mean() if asr.any() else s.sum() * 0, kl[nat].mean() if nat.any() else s.sum() * 0]
    for groups, G in ((b.dec_group, 3), (b.turn_group, 2)):
        g = torch.tensor(groups.astype(np.int64))
        means = [kl[nat & (g == k)].mean() for k in range(G) if bool((nat & (g == k)).any())]
        terms.append(torch.stack(means).mean() if means else s.sum() * 0)
    total = sum(terms)
    total.backward()
    return [float(x) for x in terms], float(total), s.grad.numpy(), kl.detach().numpy()


@pytest.mark.parametrize("T", [1.0, 2.0])
def test_matches_torch_reference_and_autograd(T):
    b = make_distill_batch(seed=3, n_utt=2, units=4, vocab=50)
    r = distill_losses(b.student, b.teacher, b.kind, b.target, b.dec_group, b.turn_group, T)
    terms, total, grad, kl = _torch_reference(b, T)
    got = [r.losses[k] for k in ("asr", "native", "dec", "turn")]
    np.testing.assert_allclose(got, terms, rtol=1e-12, atol=1e-13)
    assert abs(r.losses["total"] - total) <= 1e-12
    nat = b.kind == KIND_NATIVE
    np.testing.assert_allclose(r.kl[nat], kl[nat], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r.grad, grad, rtol=1e-10, atol=1e-13)


def test_kl_zero_when_student_equals_extended_teacher():
    b = make_distill_batch(seed=1, n_utt=1, units=3, vocab=40)
    s = np.full_like(b.student, -1e30)
    s[:, :40] = b.teacher
    r = distill_losses(s, b.teacher, b.kind, b.target, b.dec_group, b.turn_group)
    assert np.abs(r.kl).max() <= 1e-12


def test_mass_on_added_tokens_closed_form():
    # student = teacher on V, logit a on both added tokens: p_s = p_t * Z/(Z + 2e^a),
    # so KL(P_T || P_S) = log(1 + 2 e^a / Z) with Z the teacher's partition function
    rng = np.random.default_rng(0)
    t = rng.standard_normal((5, 30))
    for a in (-3.0, 0.0, 2.5):
        s = np.concatenate([t, np.full((5, 2), a)], axis=1)
        kind = np.full(5, KIND_NATIVE, np.int8)
        r = distill_losses(s, t, kind, np.full(5, -1), np.full(5, -1), np.full(5, -1))
        want = np.log1p(2 * np.exp(a) / np.exp(t).sum(axis=1))
        np.testing.assert_allclose(r.kl, want, rtol=1e-12)


def test_uniform_student_cross_entropy_is_log_vocab():
    b = make_distill_batch(seed=2, n_utt=1, units=5, vocab=60)
    s = np.zeros_like(b.student)
    r = distill_losses(s, b.teacher, b.kind, b.target, b.dec_group, b.turn_group)
    asr = b.kind == KIND_ASR
    np.testing.assert_allclose(r.ce[asr], np.log(62.0), rtol=1e-14)
    assert abs(r.losses["asr"] - np.log(62.0)) < 1e-13


def test_row_shift_invariance_and_nonnegativity():
    b = make_distill_batch(seed=4, n_utt=2, units=3, vocab=33)
    r0 = distill_losses(b.student, b.teacher, b.kind, b.target, b.dec_group, b.turn_group)
    shift = np.random.default_rng(1).standard_normal((b.n, 1)) * 7
    r1 = distill_losses(b.student + shift, b.teacher - shift[:, :1], b.kind, b.target,
                        b.dec_group, b.turn_group)
    for k in r0.losses:
        assert abs(r0.losses[k] - r1.losses[k]) < 1e-11
    assert np.all(r0.kl >= -1e-14)


def test_group_balanced_means():
    # three native rows: two listen decisions with KL a, b and one speak with c;
    # L_dec = ((a + b)/2 + c)/2 and L_native = (a + b + c)/3; turn groups absent -> 0
    rng = np.random.default_rng(5)
    t = rng.standard_normal((3, 20))
    s = t + rng.standard_normal((3, 20))
    s = np.concatenate([s, np.full((3, 2), -5.0)], axis=1)
    kind = np.full(3, KIND_NATIVE, np.int8)
    dec = np.array([0, 0, 1], np.int8)
    turn = np.full(3, -1, np.int8)
    r = distill_losses(s, t, kind, np.full(3, -1), dec, turn)
    a, b_, c = r.kl
    assert abs(r.losses["dec"] - ((a + b_) / 2 + c) / 2) < 1e-13
    assert abs(r.losses["native"] - (a + b_ + c) / 3) < 1e-13
    assert r.losses["turn"] == 0.0
    w_ce, w_kl = row_weights(kind, dec, turn)
    np.testing.assert_allclose(w_kl, [1 / 3 + 1 / 4, 1 / 3 + 1 / 4, 1 / 3 + 1 / 2])
    assert not w_ce.any()


def test_masked_rows_carry_no_loss_or_gradient():
    b = make_distill_batch(seed=6, n_utt=1, units=4, vocab=25)
    kind = b.kind.copy()
    kind[::3] = 0
    r = distill_losses(b.student, b.teacher, kind, b.target, b.dec_group, b.turn_group)
    assert not r.grad[kind == 0].any() and not r.kl[kind == 0].any() and not r.ce[kind == 0].any()
