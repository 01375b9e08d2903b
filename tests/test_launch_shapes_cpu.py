"""Launch-shape facts the GPU tests rely on, checked on the host: the decode segment
sizes that decide which decode kernel a batch takes."""
from test_gpu_argmax import SMALL_DECODE_GRID, decode_segment


def test_decode_segments_are_the_documented_sizes():
    # fp32 greedy 6144, fp32 sampling 8192, bf16 greedy 8192, bf16 sampling 10240
    assert [decode_segment(d, s) for d, s in (("f32", False), ("f32", True), ("bf16", False),
                                              ("bf16", True))] == [6144, 8192, 8192, 10240]


def test_the_launch_shape_tests_cover_both_decode_kernels():
    # the tests tile their rows to B = 8 and B = 256 at V = 40001: the first must take the
    # half-width kernel and the second the full-width one, in every mode
    V = 40001
    for dtype in ("f32", "bf16"):
        for sample in (False, True):
            seg = decode_segment(dtype, sample)
            assert 8 * (-(-V // seg)) < SMALL_DECODE_GRID <= 256 * (-(-V // seg))
