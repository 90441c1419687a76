"""Fig. 1 of the paper (Section 3, "Algorithm Intuition") on the CPU: on the
Rosenbrock function from (-1/2, 1), Adam fed the Top-1 of the gradient
wanders off Adam's path on a longer, jagged one, and adding error feedback
brings the path back to Adam's.  The paper prints no numbers for the figure;
these checks state its qualitative claim with margins measured here."""
import numpy as np
import torch

from paper_2405_15593_amd import rosenbrock as rb


def test_gradient_is_autograd():
    rng = np.random.default_rng(3)
    for _ in range(20):
        p = torch.tensor(rng.uniform(-2, 2, 2), dtype=torch.float64, requires_grad=True)
        rb.rosenbrock(p).backward()
        assert torch.allclose(rb.gradient(p.detach()), p.grad, rtol=1e-12, atol=1e-12)


def test_error_feedback_recovers_adam_path():
    steps, lr = 5000, 1e-2
    adam = rb.run_adam(steps, lr)
    topk = rb.run_adam(steps, lr, "topk")
    ef = rb.run_adam(steps, lr, "topk_ef")
    s_adam, s_topk, s_ef = rb.summary(adam), rb.summary(topk, adam), rb.summary(ef, adam)
    # Adam and Top-1 Adam with EF both reach the optimum's neighbourhood
    assert s_adam["distance_to_optimum"] < 0.05 and s_ef["distance_to_optimum"] < 0.1
    # without EF the path is jagged: much longer than Adam's
    assert s_topk["path_length"] > 1.4 * s_adam["path_length"]
    # with EF it is about as long as Adam's and stays much closer to it
    assert abs(s_ef["path_length"] - s_adam["path_length"]) < 0.2 * s_adam["path_length"]
    assert s_ef["max_deviation_from_adam"] < 0.5 * s_topk["max_deviation_from_adam"]
