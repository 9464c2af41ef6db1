"""Plan.run's argument checks, on the CPU: each wrong tensor or weight array raises
ValueError before the library is called (CPU tensors reach the device check last, so
every other check can be exercised without a GPU)."""
import numpy as np
import pytest
import torch

from paper_2608_21157_amd import binding as B


def plan(field=False, dtype=B.F32, channels=1, batch=1):
    return B.Plan(B.make_desc(3, (4, 5, 8), batch=batch, channels=channels, dtype=dtype,
                              shape=B.BOX, radius=1, has_coeff_field=field))


def good(dtype=torch.float32, batch=1):
    return torch.zeros((batch, 4, 5, 8) if batch > 1 else (4, 5, 8), dtype=dtype)


W27 = np.zeros(27, dtype=np.float32)


def raises(p, msg, *args, **kw):
    with pytest.raises(ValueError, match=msg):
        p.run(*args, steps=1, **kw)


def test_valid_cpu_tensors_stop_at_the_device_check():
    p = plan()
    raises(p, "CUDA tensors", good(), good(), W27)
    p.close()


def test_dtype_count_and_layout_of_the_tensors():
    p = plan()
    raises(p, "dtype torch.float64", good(torch.float64), good(), W27)
    raises(p, "y has dtype", good(), good(torch.float64), W27)
    raises(p, "x has 159 elements", good().flatten()[1:], good(), W27)
    raises(p, "y has 320 elements", good(), torch.zeros(320), W27)
    raises(p, "x must be contiguous", good().transpose(1, 2), good(), W27)
    raises(p, "x must be a torch tensor", good().numpy(), good(), W27)
    p.close()


def test_batch_counts_every_volume():
    p = plan(batch=3, channels=3)
    w = np.zeros((3, 27), dtype=np.float32)
    raises(p, "x has 160 elements, the plan needs batch \\* volume = 480", good(), good(), w)
    raises(p, "CUDA tensors", good(batch=3), good(batch=3), w)
    raises(p, "coeffs has 27 values, the plan needs channels \\* npoints = 81",
           good(batch=3), good(batch=3), W27)
    p.close()


def test_weights_array():
    p = plan()
    raises(p, "coeffs has dtype float64", good(), good(), W27.astype(np.float64))
    raises(p, "coeffs has 26 values", good(), good(), W27[:26])
    raises(p, "C-contiguous", good(), good(), np.zeros(54, dtype=np.float32)[::2])
    raises(p, "numpy array", good(), good(), list(W27))
    p.close()
    p = plan(dtype=B.F64)
    raises(p, "coeffs has dtype float32", good(torch.float64), good(torch.float64), W27)
    p.close()


def test_coefficient_field_presence_and_shape():
    p = plan(field=True)
    raises(p, "needs a coefficient field", good(), good(), W27)
    raises(p, "field has dtype", good(), good(), W27, field=good(torch.float64))
    raises(p, "field has 159 elements", good(), good(), W27, field=good().flatten()[1:])
    raises(p, "CUDA tensors", good(), good(), W27, field=good())
    p.close()
    p = plan()
    raises(p, "has no coefficient field", good(), good(), W27, field=good())
    p.close()


def test_a_failed_check_is_repeated_for_the_same_objects():
    """Nothing is remembered from a failed check: the same objects fail again."""
    p = plan()
    x, y = good(), good()
    for _ in range(2):
        raises(p, "CUDA tensors", x, y, W27)
    p.close()
