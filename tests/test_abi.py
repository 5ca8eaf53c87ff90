"""C-ABI checks that need no GPU: the library loads, exports every declared
symbol, validates arguments on the host before any launch, and agrees with
the input generator on the parameter table."""
import ctypes
import os
import re
from ctypes import byref, c_int32, c_int64, c_size_t, c_void_p

import pytest

from paper_2602_12529_amd import _lib, api
from paper_2602_12529_amd import configs as C
from paper_2602_12529_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h")):
        text = open(os.path.join(ROOT, "include", h)).read()
        names |= set(re.findall(r"^\s*(?:int|const char\*)\s+(ff_\w+)\s*\(", text, re.M))
    return names


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    names = declared_symbols()
    assert len(names) >= 20
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert set(_lib._SIGS) >= names


def test_version():
    assert b"gfx950" in _lib.load().ff_version()


def _err(rc, code):
    assert rc == code, (rc, _lib.load().ff_last_error())
    assert _lib.load().ff_last_error()


def test_sde_argument_validation():
    lib = _lib.load()
    fake = c_void_p(4096)   # never dereferenced: validation fails first
    ws = c_void_p(8192)
    # time order / domain
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.6, 1.0, 1, None, 0, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, 2, 8, 1.5, 0.6, 1.0, 1, None, 0, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.4, -1.0, 1, None, 0, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.4, float("nan"), 1, None, 0, None), _lib.FF_EDOMAIN)
    # ODE step cannot produce a log-prob; log-prob recompute needs sigma > 0
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), c_void_p(24576), 2, 8, 0.5, 0.4, 0.0, 1, ws, 1 << 20, None), _lib.FF_EDOMAIN)
    _err(lib.ff_logprob(fake, fake, fake, c_void_p(24576), 2, 8, 0.5, 0.4, 0.0, 1, ws, 1 << 20, None), _lib.FF_EDOMAIN)
    # dtype, null, alias, alignment, workspace
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.4, 1.0, 7, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step(None, fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step(fake, fake, fake, fake, None, 2, 8, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step(c_void_p(4100), fake, fake, c_void_p(16384), None, 2, 8, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), c_void_p(24576), 2, 8, 0.5, 0.4, 1.0, 1, ws, 1, None), _lib.FF_EWORKSPACE)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), c_void_p(24576), 2, 8, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EWORKSPACE)
    _err(lib.ff_sde_step(fake, fake, fake, c_void_p(16384), None, -1, 8, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    # empty batch is a no-op
    assert lib.ff_sde_step(None, None, None, None, None, 0, 8, 0.5, 0.4, 1.0, 1, None, 0, None) == 0
    # empty samples: only logp is touched, and it is still validated (without logp: a no-op)
    assert lib.ff_sde_step(None, None, None, None, None, 2, 0, 0.5, 0.4, 1.0, 1, None, 0, None) == 0
    _err(lib.ff_sde_step(None, None, None, None, c_void_p(24580), 2, 0, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_logprob(None, None, None, None, 2, 0, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_logprob(None, None, None, c_void_p(24580), 2, 0, 0.5, 0.4, 1.0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_noalloc(None, None, None, None, c_void_p(24580), 2, 0, 0.5, 0.4, 1.0, 1, None), _lib.FF_EINVAL)
    n = c_size_t()
    assert lib.ff_sde_workspace_size(8, 12582912, byref(n)) == 0 and n.value >= 8 * 8
    assert lib.ff_sde_workspace_size(0, 5, byref(n)) == 0 and n.value == 0


def test_sde_noalloc_argument_validation():
    """The allocation-free SDE step validates like ff_sde_step, before any device call."""
    lib = _lib.load()
    fake = c_void_p(4096)
    out, lp = c_void_p(16384), c_void_p(24576)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, out, None, 2, 8, 0.5, 0.6, 1.0, 1, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, out, lp, 2, 8, 0.5, 0.4, 0.0, 1, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, out, None, 2, 8, 0.5, 0.4, 1.0, 7, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_noalloc(None, fake, fake, out, None, 2, 8, 0.5, 0.4, 1.0, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, fake, None, 2, 8, 0.5, 0.4, 1.0, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, out, c_void_p(24580), 2, 8, 0.5, 0.4, 1.0, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_noalloc(fake, fake, fake, out, None, 70000, 8, 0.5, 0.4, 1.0, 1, None), _lib.FF_EUNSUPPORTED)
    assert lib.ff_sde_step_noalloc(None, None, None, None, None, 0, 8, 0.5, 0.4, 1.0, 1, None) == 0


def test_stream_probe_argument_validation():
    lib = _lib.load()
    fake = c_void_p(4096)
    _err(lib.ff_stream_probe(3, 1, fake, fake, 1024, 64, None), _lib.FF_EINVAL)      # mode
    _err(lib.ff_stream_probe(2, 1, fake, fake, 1000, 64, None), _lib.FF_EINVAL)      # bytes % 16
    _err(lib.ff_stream_probe(2, 1, fake, fake, 1024, 0, None), _lib.FF_EINVAL)       # blocks
    _err(lib.ff_stream_probe(0, 1, None, fake, 1024, 64, None), _lib.FF_EINVAL)      # read needs src
    _err(lib.ff_stream_probe(2, 1, c_void_p(4100), fake, 1024, 64, None), _lib.FF_EINVAL)
    assert lib.ff_stream_probe(2, 1, None, None, 0, 64, None) == 0


def test_row_classes_argument_validation():
    lib = _lib.load()
    fake = c_void_p(4096)
    _err(lib.ff_row_classes(fake, -1, 8, fake, None), _lib.FF_EINVAL)
    _err(lib.ff_row_classes(fake, 4, 0, fake, None), _lib.FF_EINVAL)
    _err(lib.ff_row_classes(None, 4, 8, fake, None), _lib.FF_EINVAL)
    _err(lib.ff_row_classes(fake, 4, 8, None, None), _lib.FF_EINVAL)
    _err(lib.ff_row_classes(fake, 4, 6, fake, None), _lib.FF_EUNSUPPORTED)          # H % 4
    _err(lib.ff_row_classes(c_void_p(4100), 4, 8, fake, None), _lib.FF_EUNSUPPORTED)  # alignment
    assert lib.ff_row_classes(None, 0, 8, None, None) == 0


def test_philox_argument_validation():
    lib = _lib.load()
    f = c_void_p(8192)
    _err(lib.ff_sde_step_philox(f, f, c_void_p(16384), None, 2, 8, 0.5, 0.6, 1.0, 1, 0, 1, None, 0, None), _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step_philox(f, f, f, None, 2, 8, 0.5, 0.4, 1.0, 1, 0, 1, None, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_sde_step_philox(f, f, c_void_p(16384), c_void_p(24576), 2, 8, 0.5, 0.4, 0.0, 1, 0, 1, None, 0, None),
         _lib.FF_EDOMAIN)
    _err(lib.ff_sde_step_philox(f, f, c_void_p(16384), c_void_p(24576), 2, 8, 0.5, 0.4, 1.0, 1, 0, 1, None, 0, None),
         _lib.FF_EWORKSPACE)
    _err(lib.ff_philox_normal(f, 2, 8, 1, 0, 4, None), _lib.FF_EINVAL)
    _err(lib.ff_philox_normal(None, 2, 8, 1, 0, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_philox4x32(None, 4, 0, 0, 0, 0, None), _lib.FF_EINVAL)
    _err(lib.ff_philox4x32(f, -1, 0, 0, 0, 0, None), _lib.FF_EINVAL)


def test_loss_argument_validation():
    """Host-side checks of the objectives: every rejected call returns before any launch."""
    lib = _lib.load()
    f = c_void_p(8192)
    ws = c_void_p(1 << 20)
    n = c_size_t()
    assert lib.ff_loss_workspace_size(4, 1000, byref(n)) == 0 and n.value >= 4 * 8
    _err(lib.ff_loss_workspace_size(-1, 8, byref(n)), _lib.FF_EINVAL)
    # noising: bad dtype, null, aliasing output, misaligned
    _err(lib.ff_flow_noise(f, f, f, c_void_p(16384), 2, 8, 5, None), _lib.FF_EINVAL)
    _err(lib.ff_flow_noise(None, f, f, c_void_p(16384), 2, 8, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_flow_noise(f, c_void_p(16384), f, c_void_p(16384), 2, 8, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_flow_noise(c_void_p(8194), f, f, c_void_p(16384), 2, 8, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_flow_noise(f, f, f, c_void_p(16384), 70000, 8, 1, None), _lib.FF_EUNSUPPORTED)
    # matching losses: workspace, null loss, null v_neg
    _err(lib.ff_awm_loss(f, f, f, f, 4, 1000, 1, None, f, None, 0, None), _lib.FF_EWORKSPACE)
    _err(lib.ff_awm_loss(f, f, f, f, 4, 1000, 1, None, f, ws, 8, None), _lib.FF_EWORKSPACE)
    _err(lib.ff_awm_loss(f, f, f, f, 4, 1000, 1, None, None, ws, 1 << 20, None), _lib.FF_EINVAL)
    _err(lib.ff_nft_loss(f, None, f, f, f, 4, 1000, 1, None, f, ws, 1 << 20, None), _lib.FF_EINVAL)
    _err(lib.ff_nft_loss(f, f, f, f, f, 4, 1000, 9, None, f, ws, 1 << 20, None), _lib.FF_EINVAL)
    assert lib.ff_awm_loss(f, f, f, f, 0, 1000, 1, None, f, None, 0, None) == 0   # empty batch: no-op
    # GRPO objective: clip range, sizes, nulls
    _err(lib.ff_grpo_loss(f, f, f, None, 8, 3, 0.0, f, None, None), _lib.FF_EDOMAIN)
    _err(lib.ff_grpo_loss(f, f, f, None, 8, 3, float("nan"), f, None, None), _lib.FF_EDOMAIN)
    _err(lib.ff_grpo_loss(f, f, f, None, 0, 3, 0.2, f, None, None), _lib.FF_EINVAL)
    _err(lib.ff_grpo_loss(f, f, f, None, 40000, 3, 0.2, f, None, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_grpo_loss(f, f, f, None, 2 ** 62, 4, 0.2, f, None, None), _lib.FF_EUNSUPPORTED)   # S*B would wrap
    _err(lib.ff_grpo_loss(None, f, f, None, 8, 3, 0.2, f, None, None), _lib.FF_EINVAL)


def test_fp8_argument_validation():
    """Host-side checks of the FP8 quantiser and linear layer: rejected calls return before any launch."""
    lib = _lib.load()
    f = c_void_p(8192)
    # quantiser: dtype, nulls, strides below the row, widths not a multiple of 8, misalignment, empty
    _err(lib.ff_quantize_fp8(f, 64, f, 64, f, 4, 64, 7, None), _lib.FF_EINVAL)
    _err(lib.ff_quantize_fp8(None, 64, f, 64, f, 4, 64, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_quantize_fp8(f, 32, f, 64, f, 4, 64, 1, None), _lib.FF_EINVAL)
    _err(lib.ff_quantize_fp8(f, 60, f, 60, f, 4, 60, 1, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_quantize_fp8(c_void_p(8200), 64, f, 64, f, 4, 64, 1, None), _lib.FF_EINVAL)
    assert lib.ff_quantize_fp8(f, 64, f, 64, f, 0, 64, 1, None) == 0
    # linear: K % 128, epilogue kind, nulls, strides, alignment, empty
    args = dict(A=f, lda=256, d_a=f, W=f, ldw=256, d_w=f, bias=None, out=f, ldo=64, M=8, N=64, K=256, epi=0)

    def call(**kw):
        a = {**args, **kw}
        return lib.ff_linear_fp8(a["A"], a["lda"], a["d_a"], a["W"], a["ldw"], a["d_w"], a["bias"], a["out"],
                                 a["ldo"], a["M"], a["N"], a["K"], a["epi"], 0, None)
    _err(call(K=192, lda=192, ldw=192), _lib.FF_EUNSUPPORTED)
    _err(call(epi=2), _lib.FF_EINVAL)
    _err(call(d_a=None), _lib.FF_EINVAL)
    _err(call(lda=128), _lib.FF_EINVAL)
    _err(call(lda=264), _lib.FF_EINVAL)
    _err(call(W=c_void_p(8200)), _lib.FF_EINVAL)
    _err(call(K=0), _lib.FF_EINVAL)
    assert call(M=0) == 0


def test_advantage_argument_validation():
    lib = _lib.load()
    f = c_void_p(4096)
    _err(lib.ff_group_advantage(f, f, f, 8, 0, 2, 0, 1e-4, f, None, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_group_advantage(f, f, f, 8, 17, 2, 0, 1e-4, f, None, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_group_advantage(f, f, f, 8, 1, 0, 0, 1e-4, f, None, None), _lib.FF_EINVAL)
    _err(lib.ff_group_advantage(f, f, f, 8, 1, 2, 3, 1e-4, f, None, None), _lib.FF_EINVAL)
    _err(lib.ff_group_advantage(f, f, f, 8, 1, 2, 0, -1.0, f, None, None), _lib.FF_EDOMAIN)
    _err(lib.ff_group_advantage(f, f, f, 8, 2, 4097, 1, 1e-4, f, None, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_group_advantage(None, f, f, 8, 1, 2, 0, 1e-4, f, None, None), _lib.FF_EINVAL)
    assert lib.ff_group_advantage(None, None, None, 0, 1, 2, 0, 1e-4, None, None, None) == 0
    _err(lib.ff_group_advantage(f, f, f, (1 << 20) + 1, 1, 2, 0, 1e-4, f, None, None), _lib.FF_EUNSUPPORTED)


@pytest.mark.parametrize("w", C.WORKLOADS, ids=lambda w: w.name)
def test_parameter_table_matches_generator(w):
    lib_table = api.tensor_table(w.model)
    gen_table = [(n, tuple(s)) for n, s, _ in synth.tensor_table(w.model)]
    assert lib_table == gen_table


def test_dit_validation_and_workspace_plan():
    lib = _lib.load()
    m = C.FLUX_BLOCK.model
    cfg = api.dit_config(m)
    n = c_int64()
    assert lib.ff_dit_num_tensors(byref(cfg), byref(n)) == 0
    ptrs = (c_void_p * n.value)(*[4096 * (i + 1) for i in range(n.value)])
    h = c_void_p()
    _err(lib.ff_dit_create(byref(cfg), ptrs, n.value - 1, byref(h)), _lib.FF_EINVAL)
    assert lib.ff_dit_create(byref(cfg), ptrs, n.value, byref(h)) == 0
    grid = (c_int32 * 3)(1, 64, 64)
    ws = c_size_t()
    assert lib.ff_dit_workspace_size(h, 8, grid, 512, 8, byref(ws)) == 0
    H, N = 3072, 4096 + 512
    assert ws.value >= 8 * N * H * 2 * 5          # Y, Q, K, V^T, O at least
    f = c_void_p(1 << 20)
    # hidden mode needs cond; outputs may not alias; workspace too small
    _err(lib.ff_dit_forward(h, f, c_void_p(2 << 20), None, 8, None, None, grid, 8, 512, c_void_p(3 << 20), None,
                            c_void_p(4 << 20), ws.value, None), _lib.FF_EINVAL)
    _err(lib.ff_dit_forward(h, f, c_void_p(2 << 20), None, 8, c_void_p(5 << 20), None, grid, 8, 512, f, None,
                            c_void_p(4 << 20), ws.value, None), _lib.FF_EINVAL)
    _err(lib.ff_dit_forward(h, f, c_void_p(2 << 20), None, 8, c_void_p(5 << 20), None, grid, 8, 512,
                            c_void_p(3 << 20), None, c_void_p(4 << 20), ws.value - 1, None), _lib.FF_EWORKSPACE)
    bad = (c_int32 * 3)(1, 63, 63)
    _err(lib.ff_dit_forward(h, f, c_void_p(2 << 20), None, 8, c_void_p(5 << 20), None, bad, 8, 512,
                            c_void_p(3 << 20), None, c_void_p(4 << 20), ws.value, None), _lib.FF_EUNSUPPORTED)
    # the prepared WAN text context: other models are rejected before any launch
    cs = c_size_t()
    _err(lib.ff_dit_context_size(h, 8, 512, byref(cs)), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_dit_context_size(None, 8, 512, byref(cs)), _lib.FF_EINVAL)
    _err(lib.ff_dit_prepare_context(h, c_void_p(2 << 20), None, 8, grid, 8, 512, c_void_p(6 << 20), 1 << 30,
                                    c_void_p(4 << 20), ws.value, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_dit_forward_ctx(h, f, c_void_p(6 << 20), 1 << 30, c_void_p(7 << 20), grid, 8, 512,
                                c_void_p(3 << 20), c_void_p(4 << 20), ws.value, None), _lib.FF_EUNSUPPORTED)
    assert lib.ff_dit_destroy(h) == 0
    # bad configs
    cfg2 = api.dit_config(m.replace(heads=7))
    _err(lib.ff_dit_num_tensors(byref(cfg2), byref(n)), _lib.FF_EINVAL)
    cfg3 = api.dit_config(m.replace(rope_axes=(16, 56, 54)))
    _err(lib.ff_dit_num_tensors(byref(cfg3), byref(n)), _lib.FF_EINVAL)


def test_dit_size_limits():
    """Block counts, widths and forward shapes beyond the library's limits are refused on the host
    (the tensor table of 2^31 blocks is never built; token counts whose products would overflow a
    launch grid or a workspace size never reach a kernel)."""
    lib = _lib.load()
    m = C.FLUX_BLOCK.model
    n = c_int64()
    for bad in (m.replace(n_dual=4097), m.replace(n_single=2 ** 31 - 1), m.replace(hidden=1 << 17, heads=1024),
                m.replace(mlp_hidden=(1 << 18) + 64)):
        _err(lib.ff_dit_num_tensors(byref(api.dit_config(bad)), byref(n)), _lib.FF_EUNSUPPORTED)
    assert lib.ff_dit_num_tensors(byref(api.dit_config(m.replace(n_dual=4096))), byref(n)) == 0
    cfg = api.dit_config(m)
    assert lib.ff_dit_num_tensors(byref(cfg), byref(n)) == 0
    ptrs = (c_void_p * n.value)(*[4096 * (i + 1) for i in range(n.value)])
    h = c_void_p()
    assert lib.ff_dit_create(byref(cfg), ptrs, n.value, byref(h)) == 0
    ws = c_size_t()
    for grid, B, n_txt, n_prompts in (((1, (1 << 20) + 1, 8), 8, 512, 8),    # an axis above 2^20
                                      ((64, 1 << 15, 1 << 15), 1, 512, 1),   # 2^34 tokens
                                      ((1, 1024, 1024), 256, 512, 256),      # B x tokens above 2^27
                                      ((1, 64, 64), 8, (1 << 20) + 8, 8),    # text above 2^20
                                      ((1, 64, 64), 8, 512, 65536)):         # prompts above 65535
        _err(lib.ff_dit_workspace_size(h, B, (c_int32 * 3)(*grid), n_txt, n_prompts, byref(ws)), _lib.FF_EUNSUPPORTED)
    assert lib.ff_dit_workspace_size(h, 1, (c_int32 * 3)(21, 30, 52), 512, 1, byref(ws)) == 0
    assert lib.ff_dit_destroy(h) == 0


def test_linear_and_attention_size_limits():
    """Shapes whose strides would overflow a tile's 32-bit load offsets, or whose tile or workgroup
    counts would overflow a launch grid, are refused on the host before any launch."""
    lib = _lib.load()
    f = c_void_p(1 << 20)
    big, K = 1 << 27, 3072
    for M, N, K_, lda in ((big + 1, 64, K, K), (64, big + 1, K, K), (64, 64, (1 << 22) + 64, (1 << 22) + 64),
                          (64, 64, K, (1 << 22) + 8), (big, big, K, K)):
        _err(lib.ff_linear(f, lda, f, None, f, max(N, 64), M, N, K_, 0, 0, None, 0, None, 0, 0, 1, None, 0, None),
             _lib.FF_EUNSUPPORTED)
    _err(lib.ff_linear_fp8(f, (1 << 22) + 128, f, f, (1 << 22) + 128, f, None, f, 64, 64, 64, (1 << 22) + 128, 0, 0,
                           None), _lib.FF_EUNSUPPORTED)
    # attention: n_kv above 2^27, too many workgroups, f32 grid rows
    _err(lib.ff_attention(f, f, f, f, 1, 1, 256, big + 8, 128, 1, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_attention(f, f, f, f, 65535, 1024, 1 << 20, 64, 128, 1, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_attention(f, f, f, f, 300, 300, 64, 64, 16, 0, None), _lib.FF_EUNSUPPORTED)
    # norm rows, joint sequence length, rotation table positions; axis widths whose int32 sum would wrap
    _err(lib.ff_norm_modulate(f, f, big + 1, 3072, None, None, 0, 0, 0, 1e-6, 1, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_qk_norm_rope(f, 1, 8, 1, 128, f, f, 1e-6, None, f, f, f, big + 8, 0, 1, None), _lib.FF_EUNSUPPORTED)
    I3 = c_int32 * 3
    _err(lib.ff_rope_table(f, I3(1 << 10, 1 << 10, 1 << 10), 128, I3(16, 56, 56), 1e4, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_rope_table(f, I3(2 ** 31 - 1, 2 ** 31 - 1, 2 ** 31 - 1), 128, I3(16, 56, 56), 1e4, None),
         _lib.FF_EUNSUPPORTED)
    _err(lib.ff_rope_table(f, I3(1, 8, 8), 8, I3(2 ** 31 - 2, 2 ** 31 - 2, 12), 1e4, None), _lib.FF_EINVAL)
    n = c_int64()
    cfg = api.dit_config(C.FLUX_BLOCK.model)
    cfg.rope_axes[0], cfg.rope_axes[1], cfg.rope_axes[2] = 2 ** 31 - 2, 2 ** 31 - 2, 132
    _err(lib.ff_dit_num_tensors(byref(cfg), byref(n)), _lib.FF_EINVAL)
    # GEMV batch and quantiser rows
    _err(lib.ff_skinny_linear(f, f, None, f, 65536, 64, 64, 0, 0, 1, None, None), _lib.FF_EUNSUPPORTED)
    _err(lib.ff_quantize_fp8(f, 64, f, 64, f, big + 1, 64, 1, None), _lib.FF_EUNSUPPORTED)


def test_dit_entry_points_return_a_status_for_mutated_configs():
    """Seeded mutations of valid configurations (one to three fields set to extreme or odd values):
    every entry point returns a status, and an accepted model with an accepted shape reports a
    workspace of at least one byte per element of its [B, N_img, hidden] activations (no size
    wrapped around)."""
    import random
    lib = _lib.load()
    vals = [-2 ** 31, -7, -1, 0, 1, 2, 3, 8, 64, 128, 130, 3072, 1 << 16, (1 << 16) + 8, 2 ** 31 - 1]
    rng = random.Random(7)
    bases = [C.TINY.model, C.FLUX_BLOCK.model, C.WAN_STACK.model.replace(n_wan=2)]
    fields = [f for f, _ in _lib.DitConfig._fields_]
    accepted = 0
    for _ in range(400):
        cfg = api.dit_config(rng.choice(bases))
        for _ in range(rng.choice([1, 2, 3])):
            f = rng.choice(fields)
            if f == "rope_axes":
                cfg.rope_axes[rng.randrange(3)] = rng.choice(vals)
            elif f in ("rope_theta", "norm_eps"):
                setattr(cfg, f, rng.choice([0.0, -1.0, float("nan"), 1e300, 1e-6]))
            else:
                setattr(cfg, f, rng.choice(vals))
        n = c_int64()
        if lib.ff_dit_num_tensors(byref(cfg), byref(n)) != 0:
            continue
        h = c_void_p()
        ptrs = (c_void_p * n.value)(*[4096 * (i + 1) for i in range(n.value)])
        if lib.ff_dit_create(byref(cfg), ptrs, n.value, byref(h)) != 0:
            continue
        accepted += 1
        for _ in range(4):
            grid = (rng.choice([1, 2, 8, 64, 1 << 20]), rng.choice([1, 8, 64]), rng.choice([8, 64, 1 << 21]))
            B, n_txt = rng.choice([1, 8, 65535, 65536]), rng.choice([8, 256, 1 << 21])
            ws = c_size_t()
            if lib.ff_dit_workspace_size(h, B, (c_int32 * 3)(*grid), n_txt, B, byref(ws)) == 0:
                assert ws.value >= B * grid[0] * grid[1] * grid[2] * cfg.hidden
        assert lib.ff_dit_destroy(h) == 0
    assert accepted > 20


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    """Without the HIP library the binding raises instead of falling back to anything else."""
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "libff.so"))
    with pytest.raises(RuntimeError, match="no non-HIP implementation"):
        _lib.load()
    with pytest.raises(RuntimeError):
        api.profile_reset()


def test_c_program_uses_the_library(tmp_path):
    """The headers are plain C99 (checked with -pedantic) and a C program links libff.so and calls it:
    version, a workspace size, a model's parameter count, and an error with its message."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    lib_dir = os.path.dirname(_lib.LIB_PATH)
    src = tmp_path / "use_ff.c"
    src.write_text(r"""
#include <stdio.h>
#include <string.h>
#include "ff.h"
#include "ff_ops.h"
#include "ff_loss.h"
int main(void) {
  size_t ws = 0;
  int64_t n = 0;
  ff_dit_config c;
  memset(&c, 0, sizeof c);
  c.model = FF_MODEL_MMDIT; c.io_mode = FF_IO_HIDDEN; c.dtype = FF_BF16; c.n_dual = 2;
  c.hidden = 3072; c.heads = 24; c.head_dim = 128; c.mlp_hidden = 12288;
  c.norm_kind = FF_NORM_RMS; c.rope_axes[0] = 16; c.rope_axes[1] = 56; c.rope_axes[2] = 56;
  c.rope_theta = 10000.0; c.norm_eps = 1e-6;
  if (ff_sde_workspace_size(8, 1000, &ws) != FF_OK || ws == 0) return 1;
  if (ff_dit_num_tensors(&c, &n) != FF_OK) return 2;
  c.heads = 7;
  if (ff_dit_num_tensors(&c, &n) != FF_EINVAL || strlen(ff_last_error()) == 0) return 3;
  printf("%s %lld\n", ff_version(), (long long)n);
  return 0;
}
""")
    exe = tmp_path / "use_ff"
    inc = os.path.join(root, "include")
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", inc, str(src), "-o", str(exe),
                        "-L", lib_dir, "-lff", "-Wl,-rpath," + lib_dir], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, (out.returncode, out.stderr)
    version, n = out.stdout.strip().rsplit(maxsplit=1)
    assert version and int(n) == 2 * 2 * 12   # two dual blocks, two streams, twelve tensors per stream
