"""CPU checks of the C ABI boundary: the library loads, exports every entry
point include/mdnn.h declares, and rejects bad arguments on the host (every
case below fails validation before any GPU work, so it runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mdnn.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mdnn_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def m():
    import paper_2011_11188_amd as mdnn
    return mdnn


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ["mdnn_gemm_mixed", "mdnn_conv2d_fwd", "mdnn_conv2d_bwd_data", "mdnn_conv2d_bwd_filter",
              "mdnn_bias_act_fwd", "mdnn_bias_act_bwd", "mdnn_softmax_xent", "mdnn_sgd_update",
              "mdnn_train_step", "mdnn_cast", "mdnn_mse_loss", "mdnn_maxpool2_fwd"]:
        assert n in names


def test_library_exports_every_declared_symbol(m):
    lib = ctypes.CDLL(m.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(m.exported_symbols()) == _declared()


def test_binding_has_same_names(m):
    for n in _declared():
        if n in ("mdnn_last_error", "mdnn_version"):
            continue
        assert callable(getattr(m, n)), n


FAKE = 0x10000  # never dereferenced: every call below fails validation first


@pytest.mark.parametrize("args,status", [
    # layout, M, N, K, alpha, A, lda, B, ldb, ab, beta, C, ldc, D, ldd, d
    ((7, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 3),     # bad layout
    ((0, -1, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 2),    # negative M
    ((0, 4, 4, 4, 1.0, None, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 1),     # A NULL
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, None, 4, 0), 1),     # D NULL
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 1.0, None, 0, FAKE, 4, 0), 1),     # beta without C
    ((0, 4, 4, 8, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 3),     # lda < K
    ((1, 4, 4, 8, 1.0, FAKE, 8, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 3),     # NT: ldb < K
    ((2, 8, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 3),     # TN: lda < M
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 2, 0), 3),     # ldd < N
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 2), 4),     # f16 in, bf16 out
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 0, 0.0, None, 0, FAKE, 4, 1), 4),     # f32 in, f16 out
    ((0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 9, 0.0, None, 0, FAKE, 4, 0), 4),     # unknown dtype
    ((0, 4, 4, 4, 1.0, FAKE + 1, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0), 5),  # odd A address
])
def test_gemm_rejects_bad_arguments(m, args, status):
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_gemm_mixed(*args, stream=0)
    assert e.value.status == status
    assert m.last_error()


def test_conv_rejects_bad_arguments(m):
    sh = m.ConvShape(2, 5, 5, 8, 8, 3, 3, 1)
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_conv2d_fwd(sh, None, FAKE, 1, None, 0, FAKE, 1, stream=0)
    assert e.value.status == m.ERR_NULL
    bad = m.ConvShape(2, 2, 2, 8, 8, 7, 7, 0)              # empty output
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_conv2d_fwd(bad, FAKE, FAKE, 1, None, 0, FAKE, 1, stream=0)
    assert e.value.status == m.ERR_SHAPE
    big = m.ConvShape(256, 28, 28, 32, 32, 5, 5, 2)
    need = m.mdnn_conv2d_bwd_filter_workspace(big, 2)
    assert need > 0
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_conv2d_bwd_filter(big, FAKE, FAKE, 2, FAKE, None, FAKE, need - 4, stream=0)
    assert e.value.status == m.ERR_WORKSPACE
    assert m.mdnn_conv2d_bwd_filter_workspace(bad, 1) == 0


def test_winograd_rejects_bad_arguments(m):
    sh = m.ConvShape(2, 6, 6, 8, 8, 3, 3, 1)
    need = m.mdnn_conv2d_fwd_winograd_workspace(sh, m.F16)
    # U: 16*8*8 halves, V: 16*(2*3*3 tiles)*8 halves, M: 16*18*8 floats, 256-byte segments
    assert need == 2048 + 4608 + 9216
    assert m.mdnn_conv2d_fwd_winograd_workspace(sh, m.F32) == 0
    five = m.ConvShape(2, 6, 6, 8, 8, 5, 5, 2)
    assert m.mdnn_conv2d_fwd_winograd_workspace(five, m.F16) == 0
    cases = [((five, FAKE, FAKE, m.F16, None, 0, FAKE, m.F32, FAKE, need), m.ERR_SHAPE),
             ((sh, FAKE, FAKE, m.F32, None, 0, FAKE, m.F32, FAKE, need), m.ERR_DTYPE),
             ((sh, FAKE, FAKE, m.F16, None, 0, FAKE, m.BF16, FAKE, need), m.ERR_DTYPE),
             ((sh, None, FAKE, m.F16, None, 0, FAKE, m.F32, FAKE, need), m.ERR_NULL),
             ((sh, FAKE, FAKE, m.F16, None, 0, FAKE, m.F32, FAKE, need - 1), m.ERR_WORKSPACE),
             ((sh, FAKE, FAKE, m.F16, None, 0, FAKE, m.F32, FAKE + 16, need), m.ERR_WORKSPACE)]
    for args, status in cases:
        with pytest.raises(m.MdnnError) as e:
            m.mdnn_conv2d_fwd_winograd(*args, stream=0)
        assert e.value.status == status, args


def test_other_entry_points_reject_bad_arguments(m):
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_cast(-1, FAKE, 0, FAKE, 1, stream=0)
    assert e.value.status == m.ERR_SHAPE
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_softmax_xent(4, 2000, FAKE, 2000, FAKE, None, FAKE, FAKE, 2000, 0, stream=0)
    assert e.value.status == m.ERR_SHAPE
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_softmax_xent(4, 10, FAKE, 8, FAKE, None, FAKE, FAKE, 10, 0, stream=0)
    assert e.value.status == m.ERR_LAYOUT
    with pytest.raises(m.MdnnError) as e:   # below fp32's element alignment (4-byte alignment is accepted)
        m.mdnn_sgd_update(10, FAKE + 2, FAKE, None, None, 0, 0.1, 0.0, None, stream=0)
    assert e.value.status == m.ERR_MISALIGNED
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_sgd_update(10, FAKE, FAKE + 6, None, None, 0, 0.1, 0.0, None, stream=0)
    assert e.value.status == m.ERR_MISALIGNED
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_bias_act_bwd(4, 4, FAKE, None, 1, None, FAKE, 1, stream=0)   # ReLU needs y
    assert e.value.status == m.ERR_NULL
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_maxpool2_bwd(1, 4, 4, 2, None, None, FAKE, 1, stream=0)
    assert e.value.status == m.ERR_NULL


def test_gemm_workspace_plan(m):
    """Host-side split plan of mdnn_gemm_mixed_ws: shapes whose output is a
    few tiles over a long K ask for fp32 partials, others for nothing."""
    for dt in (m.F32, m.F16, m.BF16):
        for (mm, n, k) in [(256, 10, 1024), (70, 136, 1000), (64, 128, 784)]:
            nb = m.mdnn_gemm_workspace(dt, mm, n, k)
            assert nb > 0 and nb % (4 * mm * n) == 0, (dt, mm, n, k)
        assert m.mdnn_gemm_workspace(dt, 4096, 4096, 4096) == 0
        assert m.mdnn_gemm_workspace(dt, 64, 64, 32) == 0
        assert m.mdnn_gemm_workspace(dt, -1, 64, 1024) == 0
    # 16 tiles of 128 x 128 split for fp16; 64 fp32 tiles of 64 x 64 do not
    assert m.mdnn_gemm_workspace(m.F16, 256, 1024, 3136) > 0
    assert m.mdnn_gemm_workspace(m.F32, 256, 1024, 3136) == 0
    assert m.mdnn_gemm_workspace(7, 64, 128, 784) == 0
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_gemm_mixed_ws(7, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0, None, 0, None, 0,
                             FAKE, 1024, stream=0)
    assert e.value.status == m.ERR_LAYOUT
    # the overflow flag: a 4-byte aligned device int32 (checked before anything runs)
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_gemm_mixed_ws(0, 4, 4, 4, 1.0, FAKE, 4, FAKE, 4, 1, 0.0, None, 0, FAKE, 4, 0, None, 0, None, 0,
                             None, 0, stream=0, nonfinite=FAKE + 2)
    assert e.value.status == m.ERR_MISALIGNED


def test_conv_algorithm_choice_and_errors(m):
    """The per-layer choice never picks Winograd, picks im2col + GEMM only
    with room for its workspace, and the algorithm entry point validates
    before it runs anything."""
    cs = m.ConvShape(128, 32, 32, 64, 64, 3, 3, 1)
    need = m.mdnn_conv2d_fwd_algo_workspace(cs, m.F16, m.CONV_IM2COL_GEMM)
    assert need == 128 * 32 * 32 * 576 * 2
    assert m.mdnn_conv2d_fwd_algo_workspace(cs, m.F16, m.CONV_IMPLICIT_GEMM) == 0
    assert m.mdnn_conv2d_fwd_algo_workspace(cs, m.F16, m.CONV_WINOGRAD) == m.mdnn_conv2d_fwd_winograd_workspace(cs, m.F16)
    for shape in [cs, m.ConvShape(256, 14, 14, 32, 64, 5, 5, 2), m.ConvShape(3, 9, 7, 16, 24, 3, 3, 1)]:
        assert m.mdnn_conv2d_fwd_choose(shape, m.F16, 0) == m.CONV_IMPLICIT_GEMM
        assert m.mdnn_conv2d_fwd_choose(shape, m.F16, 1 << 40) in (m.CONV_IMPLICIT_GEMM, m.CONV_IM2COL_GEMM)
    with pytest.raises(m.MdnnError) as e:                    # unknown algorithm
        m.mdnn_conv2d_fwd_algo(cs, FAKE, FAKE, m.F16, None, 0, FAKE, m.F16, 9, None, 0, stream=0)
    assert e.value.status == m.ERR_DTYPE
    with pytest.raises(m.MdnnError) as e:                    # im2col workspace too small
        m.mdnn_conv2d_fwd_algo(cs, FAKE, FAKE, m.F16, None, 0, FAKE, m.F16, m.CONV_IM2COL_GEMM, FAKE, need - 256,
                               stream=0)
    assert e.value.status == m.ERR_WORKSPACE
    with pytest.raises(m.MdnnError) as e:                    # winograd needs a 3x3 filter
        m.mdnn_conv2d_fwd_algo(m.ConvShape(2, 8, 8, 16, 16, 5, 5, 2), FAKE, FAKE, m.F16, None, 0, FAKE, m.F16,
                               m.CONV_WINOGRAD, FAKE, 1 << 30, stream=0)
    assert e.value.status == m.ERR_SHAPE


def test_noalloc_bwd_filter_rejects_shapes_beyond_its_array(m):
    """The filter gradient without a caller workspace takes at most the fixed
    48 MiB per GPU; a larger need fails before anything runs (the pointers
    are never touched)."""
    assert m.mdnn_conv2d_bwd_filter_noalloc_max_workspace() == 48 << 20
    cs = m.ConvShape(256, 28, 28, 384, 768, 5, 5, 2)
    assert m.mdnn_conv2d_bwd_filter_workspace(cs, m.F16) > 48 << 20
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_conv2d_bwd_filter_noalloc(cs, FAKE, FAKE, m.F16, FAKE, None, stream=0)
    assert e.value.status == m.ERR_WORKSPACE
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_conv2d_bwd_filter_noalloc(cs, FAKE, FAKE, 7, FAKE, None, stream=0)
    assert e.value.status == m.ERR_DTYPE


def test_split_entry_points_reject_bad_arguments(m):
    with pytest.raises(m.MdnnError) as e:                    # scale not a power of two
        m.mdnn_split_f16(4, 4, FAKE, 4, 3.0, None, FAKE, 4, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_SHAPE
    with pytest.raises(m.MdnnError) as e:                    # negative scale
        m.mdnn_split_f16(4, 4, FAKE, 4, -2.0, None, FAKE, 4, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_SHAPE
    with pytest.raises(m.MdnnError) as e:                    # scale 0 (chosen on the device) needs scale_out
        m.mdnn_split_f16(4, 4, FAKE, 4, 0.0, None, FAKE, 4, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_NULL
    with pytest.raises(m.MdnnError) as e:                    # misaligned scale_out
        m.mdnn_split_f16(4, 4, FAKE, 4, 0.0, FAKE + 2, FAKE, 4, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_MISALIGNED
    with pytest.raises(m.MdnnError) as e:                    # ldh < cols
        m.mdnn_split_f16(4, 4, FAKE, 4, 1.0, None, FAKE, 2, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_LAYOUT
    with pytest.raises(m.MdnnError) as e:                    # misaligned x
        m.mdnn_split_f16(4, 4, FAKE + 2, 4, 1.0, None, FAKE, 4, FAKE, 4, stream=0)
    assert e.value.status == m.ERR_MISALIGNED
    need = m.mdnn_gemm_split3_workspace(64, 32, 16)
    assert need >= 2 * 64 * 16 * 2 + 2 * 16 * 32 * 2 + 64 * 32 * 4
    assert m.mdnn_gemm_split3_workspace(-1, 2, 2) == 0
    args = (0, 64, 32, 16, 1.0, FAKE, 16, 1.0, FAKE, 32, 1.0, 0.0, None, 0, FAKE, 32)
    with pytest.raises(m.MdnnError) as e:                    # workspace too small
        m.mdnn_gemm_split3(*args, FAKE, need - 256, stream=0)
    assert e.value.status == m.ERR_WORKSPACE
    with pytest.raises(m.MdnnError) as e:                    # workspace not 256-byte aligned
        m.mdnn_gemm_split3(*args, FAKE + 16, need, stream=0)
    assert e.value.status == m.ERR_WORKSPACE
    bad_scale = (0, 64, 32, 16, 1.0, FAKE, 16, 0.75, FAKE, 32, 1.0, 0.0, None, 0, FAKE, 32)
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_gemm_split3(*bad_scale, FAKE, need, stream=0)
    assert e.value.status == m.ERR_SHAPE
    with pytest.raises(m.MdnnError) as e:                    # NT: ldb < K
        m.mdnn_gemm_split3(1, 64, 32, 16, 1.0, FAKE, 16, 1.0, FAKE, 8, 1.0, 0.0, None, 0, FAKE, 32,
                           FAKE, need, stream=0)
    assert e.value.status == m.ERR_LAYOUT


def test_net_create_validates_the_chain(m):
    import workloads as W
    L = m.LayerDesc
    cfg = m.TrainCfg(m.BF16, m.LOSS_XENT, 0.01, 0.0, 0, 10)
    good = [L(m.LAYER_CONV, 1, 1, 28, 28, 32, 5, 5, 2), L(m.LAYER_MAXPOOL2, 0, 32, 28, 28, 32, 0, 0, 0),
            L(m.LAYER_FC, 1, 14 * 14 * 32, 1, 1, 64, 0, 0, 0), L(m.LAYER_FC, 0, 64, 1, 1, 10, 0, 0, 0)]
    h = m.mdnn_net_create(good, 8, cfg)
    n, ws = m.mdnn_net_sizes(h)
    assert n == 32 * 25 + 32 + 6272 * 64 + 64 + 640 + 10 and ws > 0
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_net_bind(h, FAKE, FAKE, None, None, FAKE, ws, None)       # bf16 net needs lowp_w
    assert e.value.status == m.ERR_NULL
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_train_step(h, FAKE, FAKE, FAKE, stream=0)                 # not bound
    assert e.value.status == m.ERR_STATE
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_train_graph_create(h, FAKE, FAKE, FAKE)                   # not bound
    assert e.value.status == m.ERR_STATE
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_train_graph_create(None, FAKE, FAKE, FAKE)
    assert e.value.status == m.ERR_NULL
    assert m._lib.mdnn_train_graph_create(h, FAKE, FAKE, FAKE, None) == m.ERR_NULL   # out NULL
    with pytest.raises(m.MdnnError) as e:
        m.mdnn_graph_launch(None, stream=0)
    assert e.value.status == m.ERR_NULL
    m.mdnn_graph_destroy(None)
    m.mdnn_net_destroy(h)
    bad = list(good)
    bad[2] = L(m.LAYER_FC, 1, 100, 1, 1, 64, 0, 0, 0)                     # size mismatch
    with pytest.raises(m.MdnnError):
        m.mdnn_net_create(bad, 8, cfg)
    bad = list(good)
    bad[3] = L(m.LAYER_FC, 1, 64, 1, 1, 10, 0, 0, 0)                      # last layer with ReLU
    with pytest.raises(m.MdnnError):
        m.mdnn_net_create(bad, 8, cfg)
    # the three workloads' chains are accepted and match the flat parameter counts
    for f in (W.mlp784_fp32, W.lenet_bf16, W.wide_mlp_fp16):
        c = f()
        descs = [L(l.kind, l.act, l.c_in, l.h, l.w, l.c_out, l.r, l.s, l.pad) for l in c.layers]
        tc = m.TrainCfg(DT_CODE[c.dtype], c.loss, c.lr, c.momentum, int(c.loss_scaling), c.n_classes)
        h = m.mdnn_net_create(descs, c.batch, tc)
        assert m.mdnn_net_sizes(h)[0] == c.n_params
        m.mdnn_net_destroy(h)


DT_CODE = {"f32": 0, "f16": 1, "bf16": 2}


def test_gemm_tile_override_codes():
    import paper_2011_11188_amd as m
    try:
        for code in range(6):
            assert m.mdnn_set_gemm_tile(code) == 0
        assert m.mdnn_set_gemm_tile(6) == -1
        assert m.mdnn_set_gemm_tile(-1) == -1
    finally:
        m.mdnn_set_gemm_tile(0)
