"""GPU parity of the OPD target kernels (App. C) against the float64 oracle."""
import numpy as np
import pytest

from oracle import pipo_oracle as O

pytestmark = pytest.mark.gpu

# d is a difference of two fp32 log-softmax values over up to 151936 logits:
# each log-sum-exp carries a relative error of a few 1e-7 (fp32 sums of exp
# terms), about 1e-5 at log-sum-exps near 12; 1e-4 leaves a margin of ten.
KL_TOL = 1e-4


@pytest.fixture(scope="module")
def torch():
    import torch as t
    assert t.cuda.is_available(), "GPU tests need a GPU"
    return t


def _inputs(T, V, seed, pad_frac=0.25, pad_id=None):
    """A trajectory with PAD slots, its labels (the next token; PAD slots and
    some others unscored), student logits [T][V] and teacher logits over the
    PAD-free positions."""
    rng = np.random.default_rng(seed)
    pad_id = V - 1 if pad_id is None else pad_id
    tok = rng.integers(0, V - 1, T).astype(np.int32)
    tok[rng.random(T) < pad_frac] = pad_id
    tok[0] = rng.integers(0, V - 1)          # trajectories start with a prompt token
    labels = rng.integers(0, V - 1, T).astype(np.int32)
    labels[rng.random(T) < 0.1] = -1
    Tt = int(np.count_nonzero(tok != pad_id))
    ls = (rng.standard_normal((T, V), dtype=np.float32) * 2.0)
    lt = (rng.standard_normal((Tt, V), dtype=np.float32) * 2.0)
    return tok, labels, ls, lt, pad_id


def test_opd_teacher_rows_bit_exact(torch):
    from paper_2605_27255_amd import opd_teacher_rows
    for T in (1, 63, 1024, 1025, 5000):
        tok, _, _, _, pad = _inputs(T, 8, seed=T, pad_frac=0.3)
        tok[0] = pad if T == 63 else tok[0]   # one trajectory starting with PAD: row -1
        got = opd_teacher_rows(torch.from_numpy(tok).cuda(), pad).cpu().numpy()
        np.testing.assert_array_equal(got, O.opd_teacher_rows(tok, pad))


def test_opd_targets_full_vocab(torch):
    """64 positions over the 151936-token vocabulary, teacher rows from PAD compaction."""
    from paper_2605_27255_amd import opd_teacher_rows, opd_targets
    T, V = 64, 151936
    tok, labels, ls, lt, pad = _inputs(T, V, seed=7)
    rows = O.opd_teacher_rows(tok, pad)
    d_rows = opd_teacher_rows(torch.from_numpy(tok).cuda(), pad)
    kl, alpha, sums = opd_targets(torch.from_numpy(ls).cuda(), torch.from_numpy(lt).cuda(),
                                  torch.from_numpy(labels).cuda(), d_rows)
    torch.cuda.synchronize()
    d_ref, a_ref = O.opd_targets(ls, lt, rows, labels)
    kl, alpha = kl.cpu().numpy(), alpha.cpu().numpy()
    assert np.max(np.abs(kl - d_ref)) <= KL_TOL, np.max(np.abs(kl - d_ref))
    assert np.max(np.abs(alpha - a_ref)) <= KL_TOL
    assert np.all(alpha[labels < 0] == 1) and np.all(kl[labels < 0] == 0)
    ref_sums = O.opd_loss_sums(d_ref, labels)
    got = sums.cpu().numpy()
    np.testing.assert_array_equal(got[[1, 3]], np.array(ref_sums)[[1, 3]])
    assert abs(got[0] - ref_sums[0]) <= KL_TOL * T and abs(got[2] - ref_sums[2]) <= KL_TOL * T


def test_opd_targets_paper_chunk_sampled(torch):
    """The paper's chunk: 2048 positions x 151936; every position's sums, 48
    sampled positions element by element."""
    from paper_2605_27255_amd import opd_targets
    T, V = 2048, 151936
    rng = np.random.default_rng(11)
    ls = rng.standard_normal((T, V), dtype=np.float32) * 3.0
    lt = ls + rng.standard_normal((T, V), dtype=np.float32) * 0.5    # a teacher near the student
    labels = rng.integers(0, V, T).astype(np.int32)
    kl, alpha, sums = opd_targets(torch.from_numpy(ls).cuda(), torch.from_numpy(lt).cuda(),
                                  torch.from_numpy(labels).cuda(), None)
    torch.cuda.synchronize()
    kl, alpha = kl.cpu().numpy(), alpha.cpu().numpy()
    pick = rng.choice(T, 48, replace=False)
    d_ref, a_ref = O.opd_targets(ls[pick], lt[pick], np.arange(48), labels[pick])
    assert np.max(np.abs(kl[pick] - d_ref)) <= KL_TOL
    assert np.max(np.abs(alpha[pick] - a_ref)) <= KL_TOL
    # the sums add exactly what the kernel wrote, in double
    s = sums.cpu().numpy()
    even, odd = kl[0::2].astype(np.float64), kl[1::2].astype(np.float64)
    assert s[1] == T // 2 and s[3] == T // 2
    assert abs(s[0] - even.sum()) < 1e-6 * max(1.0, abs(even.sum()))
    assert abs(s[2] - odd.sum()) < 1e-6 * max(1.0, abs(odd.sum()))


def test_opd_targets_edges(torch):
    """Identical student and teacher: d = 0, alpha = 1; no scored position;
    an empty chunk; a row outside the teacher's rows is flagged with NaN."""
    from paper_2605_27255_amd import opd_targets
    T, V = 8, 1024
    rng = np.random.default_rng(5)
    ls = torch.from_numpy(rng.standard_normal((T, V), dtype=np.float32)).cuda()
    lab = torch.from_numpy(rng.integers(0, V, T).astype(np.int32)).cuda()
    kl, alpha, _ = opd_targets(ls, ls, lab)
    assert torch.max(torch.abs(kl)).item() <= 1e-6 and torch.min(alpha).item() >= 1 - 1e-6
    none = torch.full((T,), -1, dtype=torch.int32, device="cuda")
    kl, alpha, s = opd_targets(ls, ls, none)
    assert torch.all(kl == 0) and torch.all(alpha == 1) and torch.all(s == 0)
    e = torch.empty((0, V), dtype=torch.float32, device="cuda")
    kl, alpha, s = opd_targets(e, ls, torch.empty(0, dtype=torch.int32, device="cuda"))
    assert kl.numel() == 0 and torch.all(s == 0)
    rows = torch.tensor([0, 1, 2, 3, 4, 5, 6, 9], dtype=torch.int32, device="cuda")   # 9 >= Tt = 8
    kl, alpha, _ = opd_targets(ls, ls, lab, rows)
    torch.cuda.synchronize()
    assert torch.isnan(kl[7]) and torch.isnan(alpha[7]) and not torch.isnan(kl[:7]).any()


def test_opd_targets_bf16_rows(torch):
    """bf16 logit rows: the oracle on the same bf16 values (exact in float64)."""
    from paper_2605_27255_amd import opd_targets
    T, V = 96, 151936
    tok, labels, ls, lt, pad = _inputs(T, V, seed=9)
    rows = O.opd_teacher_rows(tok, pad)
    ls_b = torch.from_numpy(ls).cuda().to(torch.bfloat16)
    lt_b = torch.from_numpy(lt).cuda().to(torch.bfloat16)
    kl, alpha, sums = opd_targets(ls_b, lt_b, torch.from_numpy(labels).cuda(),
                                  torch.from_numpy(rows.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    ls64 = ls_b.float().cpu().numpy().astype(np.float64)
    lt64 = lt_b.float().cpu().numpy().astype(np.float64)
    d_ref, a_ref = O.opd_targets(ls64, lt64, rows, labels)
    assert np.max(np.abs(kl.cpu().numpy() - d_ref)) <= KL_TOL
    assert np.max(np.abs(alpha.cpu().numpy() - a_ref)) <= KL_TOL
