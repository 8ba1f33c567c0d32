"""The C ABI as seen from the host (CPU only): exported symbols and argument checks.

Every call here fails host-side validation, which the header specifies happens
before anything is enqueued, so no GPU is touched; pointers are dummy
addresses that the library never dereferences on the host.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_05597_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "grpo.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.SO):
        from paper_2606_05597_amd.build import build
        build()
    return _lib.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\s*\*)\s+(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(["grpo_advantages", "grpo_advantages_ex", "grpo_loss_workspace_bytes",
                                           "grpo_loss_fwd_bwd", "grpo_loss_fwd_bwd_noalloc",
                                           "fused_lmhead_workspace_bytes", "fused_lmhead_grpo", "grpo_token_logp",
                                           "fused_lmhead_blocked_workspace_bytes", "fused_lmhead_grpo_blocked",
                                           "grpo_vocab_shard_stats", "grpo_loss_fwd_bwd_vocab_shard",
                                           "fused_lmhead_vocab_shard_stats_workspace_bytes",
                                           "fused_lmhead_vocab_shard_stats", "fused_lmhead_grpo_vocab_shard",
                                           "fused_lmhead_vocab_shard_logits_bytes",
                                           "fused_lmhead_token_logp_workspace_bytes", "fused_lmhead_token_logp",
                                           "grpo_status_str"])


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.check_output(["nm", "-D", "--defined-only", _lib.SO], text=True)
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings(lib):
    for code in range(-6, 1):
        s = lib.grpo_status_str(code).decode()
        assert s.startswith("GRPO_"), s
    assert "unknown" in lib.grpo_status_str(-99).decode()


def test_workspace_queries(lib):
    small = lib.grpo_loss_workspace_bytes(100, 4)
    big = lib.grpo_loss_workspace_bytes(120000, 128)
    assert 0 < small < big and big % 256 == 0
    assert lib.grpo_loss_workspace_bytes(-1, 4) == 0 and lib.grpo_loss_workspace_bytes(10, 0) == 0
    assert lib.grpo_loss_workspace_bytes(0, 4) > 0  # an empty batch still needs the header and per-trajectory tables
    T, H, V, C = 65536, 3584, 151936, 8192
    f = lib.fused_lmhead_workspace_bytes(T, H, V, C, 64)
    # at least: transposed W and h (bf16), one dlogits chunk and its transpose (bf16), the fp32 dhidden accumulator
    assert f >= 2 * V * H + 2 * H * T + 2 * 2 * T * C + 4 * T * H and f % 256 == 0
    # a single chunk needs no dhidden accumulator
    assert lib.fused_lmhead_workspace_bytes(T, H, 4096, 4096, 64) < 2 * 4096 * H + 2 * H * T + 4 * T * 4096 + 4 * T * H
    # token-blocked: W^T and W packed (V rounded to 32 and to 64), h^T, two blocks' fp16 logit terms and tile
    # partials (8 bytes per row and 256-column tile), one block's D and packed D^T ((2 + 2 + 2 + 2) bytes per
    # element of [block, V rounded to 256])
    Vp = (V + 255) // 256 * 256
    w2 = 2 * ((V + 31) // 32 * 32) * H + 2 * H * ((V + 63) // 64 * 64)
    fb = lib.fused_lmhead_blocked_workspace_bytes(T, H, V, 8192, 64)
    parts = 2 * 8192 * (Vp // 256) * 8
    assert fb >= w2 + 2 * H * T + 8 * 8192 * Vp + parts and fb % 256 == 0
    assert fb < w2 + 2 * H * T + 8 * 8192 * Vp + parts + (64 << 20)
    # one block covering T needs one buffer of terms and partials
    one = lib.fused_lmhead_blocked_workspace_bytes(8192, H, V, 8192, 64)
    assert one < w2 + 2 * H * 8192 + 6 * 8192 * Vp + parts // 2 + (64 << 20)
    # a block larger than the batch is cut to the batch (rounded up to 256 rows)
    assert lib.fused_lmhead_blocked_workspace_bytes(300, H, V, 8192, 4) == \
        lib.fused_lmhead_blocked_workspace_bytes(300, H, V, 512, 4)
    for bad in (0, 300, -256):
        assert lib.fused_lmhead_blocked_workspace_bytes(T, H, V, bad, 64) == 0


D = ctypes.c_void_p(0x100000)  # a dummy, 256-byte aligned device address


def call_loss(lib, *, T=8, V=64, ld=64, dt=_lib.GRPO_BF16, n_traj=4, G=4, n_steps=4, norm=1, k=10.0, eps_low=0.2,
              eps_high=0.2, c=3.0, gs=1.0, ng=0.0, logits=D, actions=D, behave=D, adv=D, loss=D, ws=D,
              ws_bytes=1 << 30, seg_ptrs=(D, D), dlogits=D):
    seg = _lib.Segments()
    seg.n_traj, seg.group_size, seg.n_steps = n_traj, G, n_steps
    seg.step_tok_off, seg.traj_step_off = seg_ptrs
    p = _lib.LossParams()
    p.norm, p.k, p.eps_low, p.eps_high, p.dual_clip_c, p.grad_scale, p.n_groups_total = norm, k, eps_low, eps_high, c, gs, ng
    return lib.grpo_loss_fwd_bwd(logits, dt, T, V, ld, actions, behave, None, adv, ctypes.byref(seg),
                                 ctypes.byref(p), loss, dlogits, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(actions=None), _lib.GRPO_ERR_ARG),
    (dict(behave=None), _lib.GRPO_ERR_ARG),
    (dict(adv=None), _lib.GRPO_ERR_ARG),
    (dict(loss=None), _lib.GRPO_ERR_ARG),
    (dict(logits=None), _lib.GRPO_ERR_ARG),
    (dict(seg_ptrs=(None, D)), _lib.GRPO_ERR_ARG),
    (dict(ld=63), _lib.GRPO_ERR_SHAPE),
    (dict(V=0), _lib.GRPO_ERR_SHAPE),
    (dict(T=-1), _lib.GRPO_ERR_SHAPE),
    (dict(T=1 << 31), _lib.GRPO_ERR_SHAPE),
    (dict(n_traj=6), _lib.GRPO_ERR_SHAPE),          # not a multiple of G
    (dict(n_steps=3), _lib.GRPO_ERR_SHAPE),         # fewer steps than trajectories
    (dict(G=0), _lib.GRPO_ERR_SHAPE),
    (dict(norm=7), _lib.GRPO_ERR_ARG),
    (dict(k=0.0), _lib.GRPO_ERR_ARG),               # CONST_K needs k > 0
    (dict(eps_low=1.0), _lib.GRPO_ERR_ARG),
    (dict(eps_low=-0.1), _lib.GRPO_ERR_ARG),
    (dict(eps_high=-0.1), _lib.GRPO_ERR_ARG),
    (dict(c=0.5), _lib.GRPO_ERR_ARG),               # the dual clip needs c > 1 (or 0 = off)
    (dict(c=1.0), _lib.GRPO_ERR_ARG),
    (dict(gs=float("inf")), _lib.GRPO_ERR_ARG),
    (dict(ng=-1.0), _lib.GRPO_ERR_ARG),
    (dict(dt=5), _lib.GRPO_ERR_DTYPE),
    (dict(logits=ctypes.c_void_p(0x100001)), _lib.GRPO_ERR_ALIGN),
    (dict(dlogits=ctypes.c_void_p(0x100003), dt=_lib.GRPO_F32), _lib.GRPO_ERR_ALIGN),
    (dict(ws=None), _lib.GRPO_ERR_WORKSPACE),
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
    (dict(ws=ctypes.c_void_p(0x100010)), _lib.GRPO_ERR_ALIGN),
])
def test_loss_rejects_bad_arguments(lib, kw, status):
    assert call_loss(lib, **kw) == status


def call_loss_noalloc(lib, *, T=8, V=64, ld=64, n_traj=4, G=4, n_steps=4, logits=D, actions=D):
    seg = _lib.Segments()
    seg.n_traj, seg.group_size, seg.n_steps = n_traj, G, n_steps
    seg.step_tok_off, seg.traj_step_off = D, D
    p = _lib.LossParams()
    p.norm, p.k, p.eps_low, p.eps_high, p.dual_clip_c, p.grad_scale, p.n_groups_total = 1, 10.0, 0.2, 0.2, 3.0, 1.0, 0.0
    return lib.grpo_loss_fwd_bwd_noalloc(logits, _lib.GRPO_BF16, T, V, ld, actions, D, None, D, ctypes.byref(seg),
                                         ctypes.byref(p), D, D, None, None)


def test_noalloc_rejects_bad_arguments_and_oversized_batches(lib):
    # the argument checks of grpo_loss_fwd_bwd, then the batch against the fixed scratch array, all on the host
    assert call_loss_noalloc(lib, actions=None) == _lib.GRPO_ERR_ARG
    assert call_loss_noalloc(lib, ld=63) == _lib.GRPO_ERR_SHAPE
    assert call_loss_noalloc(lib, logits=ctypes.c_void_p(0x100001)) == _lib.GRPO_ERR_ALIGN
    big_T = 1 << 20  # 61 bytes of scratch per token: 64 MB > 24 MiB
    assert lib.grpo_loss_workspace_bytes(big_T, 4) > _lib.GRPO_NOALLOC_SCRATCH_BYTES
    assert call_loss_noalloc(lib, T=big_T) == _lib.GRPO_ERR_WORKSPACE
    many = 1 << 20  # per-trajectory tables alone exceed the array
    assert call_loss_noalloc(lib, n_traj=many, G=1, n_steps=many) == _lib.GRPO_ERR_WORKSPACE
    # the sizes the header states fit
    assert lib.grpo_loss_workspace_bytes(262144, 16384) <= _lib.GRPO_NOALLOC_SCRATCH_BYTES


def test_trajectory_normaliser_ignores_k(lib):
    # k is only checked for the constant normaliser; with 1/|tau_i| a zero k passes validation
    # (a workspace that is too small then stops the call before any launch)
    assert call_loss(lib, norm=0, k=0.0, ws_bytes=16) == _lib.GRPO_ERR_WORKSPACE


def test_advantages_rejects_bad_arguments(lib):
    f = lib.grpo_advantages
    assert f(None, 8, 8, 1, 0.0, D, None) == _lib.GRPO_ERR_ARG
    assert f(D, 8, 8, 2, 0.0, D, None) == _lib.GRPO_ERR_ARG          # ddof in {0, 1}
    assert f(D, 8, 8, 1, -1.0, D, None) == _lib.GRPO_ERR_ARG         # std_eps >= 0
    assert f(D, 12, 8, 1, 0.0, D, None) == _lib.GRPO_ERR_SHAPE       # n_traj % G
    assert f(D, 0, 8, 1, 0.0, D, None) == _lib.GRPO_ERR_SHAPE


def call_fused(lib, *, blocked=False, T=8, H=64, V=512, chunk=256, hidden=D, w=D, dh=D, dw=D, ws=D,
               ws_bytes=1 << 40):
    seg = _lib.Segments()
    seg.n_traj, seg.group_size, seg.n_steps = 4, 4, 4
    seg.step_tok_off, seg.traj_step_off = D, D
    p = _lib.LossParams()
    p.norm, p.k, p.eps_low, p.eps_high, p.dual_clip_c, p.grad_scale = 1, 10.0, 0.2, 0.2, 0.0, 1.0
    args = (hidden, w, T, H, V, chunk, D, D, None, D, ctypes.byref(seg), ctypes.byref(p), D, dh, dw, 0, None, ws,
            ws_bytes, None)
    return lib.fused_lmhead_grpo_blocked(*args, None) if blocked else lib.fused_lmhead_grpo(*args)


@pytest.mark.parametrize("kw,status", [
    (dict(H=96), _lib.GRPO_ERR_SHAPE),        # H a multiple of 64
    (dict(T=(1 << 23) - 255), _lib.GRPO_ERR_SHAPE),  # T- and V-long operand rows addressed with 32-bit offsets
    (dict(V=(1 << 23) - 248), _lib.GRPO_ERR_SHAPE),
    (dict(V=500), _lib.GRPO_ERR_SHAPE),       # V a multiple of 8
    (dict(chunk=300), _lib.GRPO_ERR_SHAPE),   # chunk a multiple of 256
    (dict(chunk=0), _lib.GRPO_ERR_SHAPE),
    (dict(w=None), _lib.GRPO_ERR_ARG),
    (dict(dw=None), _lib.GRPO_ERR_ARG),
    (dict(hidden=None), _lib.GRPO_ERR_ARG),
    (dict(dh=ctypes.c_void_p(0x100008)), _lib.GRPO_ERR_ALIGN),
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
])
@pytest.mark.parametrize("blocked", [False, True])
def test_fused_rejects_bad_arguments(lib, kw, status, blocked):
    # chunk: the vocabulary chunk, or for the token-blocked entry the token block (same rule: a multiple of 256)
    assert call_fused(lib, blocked=blocked, **kw) == status


def test_fused_blocked_rejects_oversized_block(lib):
    assert call_fused(lib, blocked=True, chunk=1 << 23) == _lib.GRPO_ERR_SHAPE


def call_logp(lib, *, logits=D, dt=_lib.GRPO_BF16, T=8, V=64, ld=64, actions=D):
    return lib.grpo_token_logp(logits, dt, T, V, ld, actions, D, D, None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(logits=None), _lib.GRPO_ERR_ARG),
    (dict(actions=None), _lib.GRPO_ERR_ARG),
    (dict(T=-1), _lib.GRPO_ERR_SHAPE),
    (dict(T=1 << 31), _lib.GRPO_ERR_SHAPE),
    (dict(V=0), _lib.GRPO_ERR_SHAPE),
    (dict(ld=63), _lib.GRPO_ERR_SHAPE),
    (dict(dt=7), _lib.GRPO_ERR_DTYPE),
    (dict(logits=ctypes.c_void_p(0x100001)), _lib.GRPO_ERR_ALIGN),
    (dict(logits=ctypes.c_void_p(0x100002), dt=_lib.GRPO_F32), _lib.GRPO_ERR_ALIGN),
])
def test_token_logp_rejects_bad_arguments(lib, kw, status):
    assert call_logp(lib, **kw) == status


def call_shard_stats(lib, *, logits=D, dt=_lib.GRPO_BF16, T=8, V=64, ld=64, v_begin=0, actions=D, stats=D):
    return lib.grpo_vocab_shard_stats(logits, dt, T, V, ld, v_begin, actions, stats, None, None)


@pytest.mark.parametrize("kw,status", [
    (dict(logits=None), _lib.GRPO_ERR_ARG),
    (dict(actions=None), _lib.GRPO_ERR_ARG),
    (dict(stats=None), _lib.GRPO_ERR_ARG),
    (dict(T=-1), _lib.GRPO_ERR_SHAPE),
    (dict(V=0), _lib.GRPO_ERR_SHAPE),
    (dict(ld=63), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=-8), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=(1 << 31) - 64), _lib.GRPO_ERR_SHAPE),  # the shard's last column past 2^31
    (dict(dt=3), _lib.GRPO_ERR_DTYPE),
    (dict(logits=ctypes.c_void_p(0x100001)), _lib.GRPO_ERR_ALIGN),
    (dict(stats=ctypes.c_void_p(0x100004)), _lib.GRPO_ERR_ALIGN),  # records are 8-byte aligned
])
def test_shard_stats_rejects_bad_arguments(lib, kw, status):
    assert call_shard_stats(lib, **kw) == status


def call_shard_loss(lib, *, T=8, V=64, ld=64, v_begin=0, V_total=128, stats=D, n_shards=2, logits=D, dlogits=D,
                    dt=_lib.GRPO_BF16, ws=D, ws_bytes=1 << 30):
    seg = _lib.Segments()
    seg.n_traj, seg.group_size, seg.n_steps = 4, 4, 4
    seg.step_tok_off, seg.traj_step_off = D, D
    p = _lib.LossParams()
    p.norm, p.k, p.eps_low, p.eps_high, p.dual_clip_c, p.grad_scale = 1, 10.0, 0.2, 0.2, 0.0, 1.0
    return lib.grpo_loss_fwd_bwd_vocab_shard(logits, dt, T, V, ld, v_begin, V_total, stats, n_shards, D, D, None, D,
                                             ctypes.byref(seg), ctypes.byref(p), D, dlogits, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(logits=None), _lib.GRPO_ERR_ARG),
    (dict(stats=None), _lib.GRPO_ERR_ARG),
    (dict(V=0), _lib.GRPO_ERR_SHAPE),
    (dict(ld=63), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=-1), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=72), _lib.GRPO_ERR_SHAPE),          # v_begin + V_shard > V_total
    (dict(V_total=1 << 31), _lib.GRPO_ERR_SHAPE),
    (dict(n_shards=0), _lib.GRPO_ERR_SHAPE),
    (dict(n_shards=65537), _lib.GRPO_ERR_SHAPE),
    (dict(dt=9), _lib.GRPO_ERR_DTYPE),
    (dict(stats=ctypes.c_void_p(0x100004)), _lib.GRPO_ERR_ALIGN),
    (dict(dlogits=ctypes.c_void_p(0x100001)), _lib.GRPO_ERR_ALIGN),
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
])
def test_shard_loss_rejects_bad_arguments(lib, kw, status):
    assert call_shard_loss(lib, **kw) == status


def call_fused_shard_stats(lib, *, T=8, H=64, V=512, v_begin=0, hidden=D, w=D, stats=D, logits=None, ws=D,
                           ws_bytes=1 << 30):
    return lib.fused_lmhead_vocab_shard_stats(hidden, w, T, H, V, v_begin, D, stats, logits, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=96), _lib.GRPO_ERR_SHAPE),
    (dict(V=500), _lib.GRPO_ERR_SHAPE),
    (dict(T=-1), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=-8), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=(1 << 31) - 512), _lib.GRPO_ERR_SHAPE),
    (dict(w=None), _lib.GRPO_ERR_ARG),
    (dict(hidden=None), _lib.GRPO_ERR_ARG),
    (dict(stats=None), _lib.GRPO_ERR_ARG),
    (dict(stats=ctypes.c_void_p(0x100004)), _lib.GRPO_ERR_ALIGN),
    (dict(logits=ctypes.c_void_p(0x100008)), _lib.GRPO_ERR_ALIGN),  # the kept logits are 16-byte aligned
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
])
def test_fused_shard_stats_rejects_bad_arguments(lib, kw, status):
    assert call_fused_shard_stats(lib, **kw) == status


def test_fused_shard_stats_workspace(lib):
    T, H, Vs = 65536, 3584, 18992
    n = lib.fused_lmhead_vocab_shard_stats_workspace_bytes(T, H, Vs)
    assert n >= 2 * Vs * H + 8 * T * ((Vs + 255) // 256) and n % 256 == 0
    assert lib.fused_lmhead_vocab_shard_stats_workspace_bytes(-1, H, Vs) == 0
    # the kept logits: fp32, T and V_shard rounded up to the 256 tile
    assert lib.fused_lmhead_vocab_shard_logits_bytes(T, Vs) == 4 * T * 19200
    assert lib.fused_lmhead_vocab_shard_logits_bytes(300, 8) == 4 * 512 * 256
    assert lib.fused_lmhead_vocab_shard_logits_bytes(-1, Vs) == 0 and lib.fused_lmhead_vocab_shard_logits_bytes(T, 0) == 0


def call_fused_shard(lib, *, T=8, H=64, V=512, v_begin=0, V_total=1024, chunk=256, stats=D, n_shards=2, hidden=D,
                     w=D, dhp=D, dw=D, logits=None, ws=D, ws_bytes=1 << 40):
    seg = _lib.Segments()
    seg.n_traj, seg.group_size, seg.n_steps = 4, 4, 4
    seg.step_tok_off, seg.traj_step_off = D, D
    p = _lib.LossParams()
    p.norm, p.k, p.eps_low, p.eps_high, p.dual_clip_c, p.grad_scale = 1, 10.0, 0.2, 0.2, 0.0, 1.0
    return lib.fused_lmhead_grpo_vocab_shard(hidden, w, T, H, V, v_begin, V_total, chunk, stats, n_shards, D, D, None,
                                             D, ctypes.byref(seg), ctypes.byref(p), D, dhp, dw, 0, None, logits, ws,
                                             ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=96), _lib.GRPO_ERR_SHAPE),
    (dict(V=500), _lib.GRPO_ERR_SHAPE),
    (dict(T=(1 << 23) - 255), _lib.GRPO_ERR_SHAPE),
    (dict(chunk=300), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=-8), _lib.GRPO_ERR_SHAPE),
    (dict(v_begin=520), _lib.GRPO_ERR_SHAPE),      # v_begin + V_shard > V_total
    (dict(V_total=1 << 31), _lib.GRPO_ERR_SHAPE),
    (dict(n_shards=0), _lib.GRPO_ERR_SHAPE),
    (dict(w=None), _lib.GRPO_ERR_ARG),
    (dict(dw=None), _lib.GRPO_ERR_ARG),
    (dict(dhp=None), _lib.GRPO_ERR_ARG),
    (dict(stats=None), _lib.GRPO_ERR_ARG),
    (dict(dhp=ctypes.c_void_p(0x100008)), _lib.GRPO_ERR_ALIGN),
    (dict(stats=ctypes.c_void_p(0x100004)), _lib.GRPO_ERR_ALIGN),
    (dict(logits=ctypes.c_void_p(0x100008)), _lib.GRPO_ERR_ALIGN),
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
])
def test_fused_shard_rejects_bad_arguments(lib, kw, status):
    assert call_fused_shard(lib, **kw) == status


def test_fused_shard_kept_logits_ignores_chunk(lib):
    # with the statistics call's logits the shard is one chunk: a chunk that is not a multiple of 256 passes the
    # shape checks, and the workspace needed is the whole-shard chunk's (T = 8, H = 64, V_shard = 512, 4 trajectories)
    assert call_fused_shard(lib, chunk=300) == _lib.GRPO_ERR_SHAPE
    need = lib.fused_lmhead_workspace_bytes(8, 64, 512, 512, 4)
    assert call_fused_shard(lib, chunk=300, logits=D, ws_bytes=need - 1) == _lib.GRPO_ERR_WORKSPACE


def test_advantages_ex_rejects_bad_arguments(lib):
    f = lib.grpo_advantages_ex
    assert f(D, 8, 8, 2, 1, 0.0, D, None, None, None) == _lib.GRPO_ERR_ARG       # unknown mode
    assert f(D, 8, 8, -1, 1, 0.0, D, None, None, None) == _lib.GRPO_ERR_ARG
    assert f(None, 8, 8, 0, 1, 0.0, D, None, None, None) == _lib.GRPO_ERR_ARG
    assert f(D, 8, 8, 1, 1, 0.0, None, None, None, None) == _lib.GRPO_ERR_ARG
    assert f(D, 8, 8, 1, 3, 0.0, D, None, None, None) == _lib.GRPO_ERR_ARG      # ddof checked under the filter too
    assert f(D, 12, 8, 1, 1, 0.0, D, None, None, None) == _lib.GRPO_ERR_SHAPE
    assert f(D, 0, 1, 1, 1, 0.0, D, None, None, None) == _lib.GRPO_ERR_SHAPE


def call_fused_logp(lib, *, T=8, H=64, V=512, hidden=D, w=D, actions=D, logp=D, ent=D, ws=D, ws_bytes=1 << 30):
    return lib.fused_lmhead_token_logp(hidden, w, T, H, V, actions, logp, ent, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(H=96), _lib.GRPO_ERR_SHAPE),
    (dict(V=500), _lib.GRPO_ERR_SHAPE),
    (dict(T=-1), _lib.GRPO_ERR_SHAPE),
    (dict(T=(1 << 23) - 255), _lib.GRPO_ERR_SHAPE),
    (dict(w=None), _lib.GRPO_ERR_ARG),
    (dict(hidden=None), _lib.GRPO_ERR_ARG),
    (dict(actions=None), _lib.GRPO_ERR_ARG),
    (dict(hidden=ctypes.c_void_p(0x100008)), _lib.GRPO_ERR_ALIGN),
    (dict(logp=ctypes.c_void_p(0x100002)), _lib.GRPO_ERR_ALIGN),
    (dict(ws_bytes=16), _lib.GRPO_ERR_WORKSPACE),
])
def test_fused_logp_rejects_bad_arguments(lib, kw, status):
    assert call_fused_logp(lib, **kw) == status


def test_fused_logp_workspace(lib):
    T, H, V = 65536, 3584, 151936
    n = lib.fused_lmhead_token_logp_workspace_bytes(T, H, V)
    assert n >= 2 * V * H + 12 * T * 594 and n % 256 == 0
    assert lib.fused_lmhead_token_logp_workspace_bytes(-1, H, V) == 0
