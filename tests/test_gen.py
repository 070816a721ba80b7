"""The seeded generator: row blocks equal the full draw; distributions as stated."""
import numpy as np

from gen import MatrixSpec, workload_matrices, gen_matrix, gen_x, bf16_bits_to_f32


def test_row_block_equals_full_draw():
    spec = MatrixSpec(4, 0, 1, "k", 64, 256, layer_scale=True)
    full = gen_matrix(spec)
    assert np.array_equal(gen_matrix(spec, slice(10, 30)), full[10:30])
    spec2 = MatrixSpec(2, 0, 0, "q", 48, 128, row_scale=True)
    assert np.array_equal(gen_matrix(spec2, slice(5, 48)), gen_matrix(spec2)[5:48])


def test_config_shapes():
    assert [(m.rows, m.cols) for m in workload_matrices(4)] == [
        (4096, 4096), (1024, 4096), (1024, 4096), (4096, 4096),
        (14336, 4096), (14336, 4096), (4096, 14336)]
    assert sum(m.rows * m.cols for m in workload_matrices(5)) * 80 == 68451041280


def test_distribution_workload1():
    spec = workload_matrices(1)[0]
    w = bf16_bits_to_f32(gen_matrix(spec)).astype(np.float64)
    assert abs(w.std() - 0.02 * np.sqrt(1 + 0.001 * 399)) < 2e-3
    big = np.abs(w) > 0.2
    assert 0.0003 < big.mean() < 0.0015
    x = gen_x(spec, 1, "f32")
    assert x.shape == (1, 1024) and x.dtype == np.float32


def test_thread_count_and_block_boundaries():
    spec = MatrixSpec(3, 0, 2, "down", 600, 64)
    a = gen_matrix(spec, threads=1)
    assert np.array_equal(a, gen_matrix(spec, threads=5))
    assert np.array_equal(gen_matrix(spec, slice(250, 530), threads=3), a[250:530])
