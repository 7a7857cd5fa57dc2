"""Host logic of the eps-selection protocol (Sec. IV-B): start at 0.1, divide
by 10 until the training accuracy exceeds 97%, else take the first eps whose
accuracy agrees with the next one in three digits."""
from paper_2202_12674_amd.eps_sweep import DEFAULT_EPS, tune_eps


def rows(accs):
    return [{"eps": 10.0 ** (-(k + 1)), "train_acc": a} for k, a in enumerate(accs)]


def test_default_grid():
    assert DEFAULT_EPS[0] == 0.1 and len(DEFAULT_EPS) == 15
    assert all(abs(b / a - 0.1) < 1e-12 for a, b in zip(DEFAULT_EPS, DEFAULT_EPS[1:]))


def test_first_eps_above_target():
    assert tune_eps(rows([0.5, 0.9, 0.971, 0.99])) == (1e-3, "accuracy above target")


def test_exactly_target_is_not_above():
    assert tune_eps(rows([0.5, 0.97, 0.969, 0.975]))[0] == 1e-4


def test_settled_in_three_digits():
    eps, why = tune_eps(rows([0.5, 0.9021, 0.9026, 0.9027]))
    assert (eps, why) == (1e-2, "accuracy settled in three digits")


def test_fallback_smallest():
    assert tune_eps(rows([0.5, 0.6, 0.7])) == (1e-3, "smallest eps")
