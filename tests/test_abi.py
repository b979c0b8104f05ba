"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/bt.h declares, computes the flat parameter layout of the seeded
generator, and rejects bad arguments before launching anything."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_24780_amd import bt, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bt.h")

BT_OK, BT_EINVAL, BT_ESHAPE, BT_EALIGN, BT_EWORKSPACE = 0, 1, 2, 3, 4
FAKE = 0x10000      # 16-byte aligned, never dereferenced: validation fails first
FAKE_MIS = 0x10004  # misaligned


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bt_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bt.LIB_PATH):
        pytest.fail("libbt.so is not built (run python -m paper_2606_24780_amd.build)")
    return bt.lib()


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert len(names) >= 30
    raw = ctypes.CDLL(bt.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), f"libbt.so does not export {n}"
    assert set(names) == set(bt.EXPORTED), set(names) ^ set(bt.EXPORTED)


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(bt, "_lib", None)
    monkeypatch.setattr(bt, "LIB_PATH", "/nonexistent/libbt.so")
    with pytest.raises(bt.BTLibraryError):
        bt.lib()


@pytest.mark.parametrize("cfg", [synth.TINY, synth.GPT2_124M, synth.GPT2Config(V=50, Vp=56, max_T=8, L=3, H=2, C=16)])
def test_param_layout_matches_generator(lib, cfg):
    hp = synth.HP_124M
    assert bt.num_params(cfg, hp) == synth.num_params(cfg)
    assert lib.bt_gpt2_num_decay_params(ctypes.byref(bt.make_config(cfg, hp))) == synth.num_decay_params(cfg)
    assert bt.param_offsets(cfg, hp) == synth.param_offsets(cfg)
    assert all(o % 4 == 0 for o in synth.param_offsets(cfg))


def test_status_strings(lib):
    assert lib.bt_status_str(BT_ESHAPE) == b"BT_ESHAPE"
    assert lib.bt_version().decode().count(".") == 2


def _gemm(lib, opA=0, opB=0, M=128, N=128, K=128, A=FAKE, lda=128, B=FAKE, ldb=128, beta=0.0, C=FAKE,
          ldc=128, bias=None, epi=0, pre=None, gin=None, res=None, cs=None, ws=None, wsb=0):
    return lib.bt_gemm(opA, opB, M, N, K, A, lda, B, ldb, beta, C, ldc, bias, epi, pre, gin, res, cs, ws, wsb,
                       None)


def test_gemm_validation(lib):
    assert _gemm(lib, M=130) == BT_ESHAPE
    assert _gemm(lib, lda=64) == BT_ESHAPE
    assert _gemm(lib, A=FAKE_MIS) == BT_EALIGN
    assert _gemm(lib, beta=0.5) == BT_EINVAL
    assert _gemm(lib, epi=1) == BT_EINVAL           # bias missing
    assert _gemm(lib, epi=3) == BT_EINVAL           # gelu_in missing
    assert _gemm(lib, res=FAKE) == BT_EINVAL        # residual aliases C
    assert _gemm(lib, opA=5) == BT_EINVAL
    assert _gemm(lib, C=None) == BT_EINVAL
    assert _gemm(lib, opB=1, cs=FAKE + 4096) == BT_EINVAL   # column sums need op(B) = B
    assert _gemm(lib, epi=1, bias=FAKE, cs=FAKE + 4096) == BT_EINVAL
    assert b"multiples of 4" in lib.bt_last_error() or True
    # a split-K shape without workspace
    need = lib.bt_gemm_ws_bytes(1, 0, 768, 768, 16384, 0)
    assert need > 0
    assert _gemm(lib, opA=1, M=768, N=768, K=16384, lda=768, ldb=768, ldc=768) == BT_EWORKSPACE
    # an epilogue product with a long K splits too (the epilogue runs in the reduction)
    need = lib.bt_gemm_ws_bytes(0, 0, 256, 256, 4096, 1)
    assert need > 0
    assert _gemm(lib, M=256, N=256, K=4096, lda=4096, ldb=256, ldc=256, epi=1, bias=FAKE + 4096, ws=FAKE + 8192,
                 wsb=need - 1) == BT_EWORKSPACE
    assert _gemm(lib, M=0) == BT_OK                  # empty product: nothing to do


def test_other_validation(lib):
    assert lib.bt_attention_fwd(FAKE, FAKE, FAKE, 1, 16, 1, 132, None) == BT_ESHAPE
    assert lib.bt_attention_fwd(FAKE, FAKE, FAKE, 0, 16, 1, 64, None) == BT_ESHAPE
    assert lib.bt_attention_bwd(FAKE, FAKE, FAKE, FAKE, FAKE + 4096, None, 0, 1, 16, 1, 64, None) == BT_EWORKSPACE
    assert lib.bt_attention_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20, 1, 16, 1, 64, None) == BT_EINVAL
    assert lib.bt_layernorm_fwd(FAKE, FAKE, FAKE, FAKE + 64, FAKE, FAKE, 4, 6, 1e-5, None) == BT_ESHAPE
    assert lib.bt_layernorm_fwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 8, 1e-5, None) == BT_EINVAL  # y aliases x
    assert lib.bt_layernorm_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1.0, 0.0, None, 0, 4, 8, None) == BT_EINVAL
    assert lib.bt_softmax_xent_fwd(FAKE, FAKE, FAKE, FAKE, 4, 10, 8, None) == BT_ESHAPE
    # the widest row the cross-entropy kernels take is 65,536 columns
    assert lib.bt_softmax_xent_fwd(FAKE, FAKE, FAKE, FAKE, 4, 65537, 65540, None) == BT_ESHAPE
    assert lib.bt_softmax_xent_fused(FAKE, FAKE, FAKE, FAKE, 1.0, 4, 65537, 65540, None) == BT_ESHAPE
    assert lib.bt_layernorm_fwd(FAKE, FAKE, FAKE, FAKE + 64, FAKE, FAKE, 4, 4100, 1e-5, None) == BT_ESHAPE
    assert lib.bt_adamw_step(FAKE, FAKE, FAKE, FAKE, 8, 4, 1e-3, 0.9, 0.95, 1e-8, 0.1, 0, None, None) == BT_EINVAL
    assert lib.bt_adamw_step(FAKE, FAKE, FAKE, FAKE, 8, 12, 1e-3, 0.9, 0.95, 1e-8, 0.1, 1, None, None) == BT_ESHAPE
    assert lib.bt_gelu_fwd(FAKE, FAKE, 6, None) == BT_ESHAPE
    assert lib.bt_colsum(FAKE, 4, 6, 8, FAKE, 0.0, None, 0, None) == BT_ESHAPE
    assert lib.bt_embedding_bwd(FAKE, FAKE, FAKE, FAKE, 0.0, None, 0, 2, 4, 8, 16, None) == BT_EWORKSPACE
    assert lib.bt_grad_norm_clip(FAKE, 8, 1.0, None, None, None, 0, None) == BT_EINVAL


def test_gemm_plan(lib):
    """bt_gemm_plan (host only) agrees with the workspace query (split exactly
    when a workspace is needed), takes the 32-deep tile for the LM head's
    input gradient (K = 50,304 over 768 tiles) and never for products with
    both operands MN-contiguous, copies full tiles directly and stages ragged
    ones, and validates its arguments."""
    shapes = [(0, 0, 16384, 768, 50304), (0, 1, 16384, 50304, 768), (1, 0, 768, 50304, 16384),
              (0, 0, 16384, 2304, 768), (1, 0, 768, 2304, 16384), (0, 0, 260, 196, 132), (1, 1, 4, 4, 4),
              (0, 1, 16384, 768, 3072), (1, 1, 1028, 2052, 8196)]
    for ta, tb, M, N, K in shapes:
        d, sp, dr = bt.bt_gemm_plan(ta, tb, M, N, K, M if ta else K, K if tb else N)
        assert d in (16, 32) and sp >= 1 and dr in (0, 1)
        assert (sp > 1) == (lib.bt_gemm_ws_bytes(ta, tb, M, N, K, 0) > 0)
        ragged = M % 128 or N % 128 or K % d
        assert dr == (0 if ragged else 1)
    assert bt.bt_gemm_plan(0, 0, 16384, 768, 50304, 50304, 768)[0] == 32
    for M, N, K in [(768, 50304, 16384), (4096, 2048, 32768), (2048, 4096, 1024), (384, 2048, 4096)]:
        assert bt.bt_gemm_plan(1, 0, M, N, K, M, N)[0] == 16
    with pytest.raises(bt.BTError) as e:
        bt.bt_gemm_plan(0, 0, 6, 4, 4, 4, 4)
    assert e.value.status == BT_ESHAPE
    d = ctypes.c_int()
    assert lib.bt_gemm_plan(0, 0, 4, 4, 4, 4, 4, ctypes.byref(d), None, ctypes.byref(d)) == BT_EINVAL


def test_attention_workspace_sizes(lib):
    """Row sums D always; the stored-dS method adds B H T T floats when T % 4 == 0."""
    def al(x):
        return (x + 255) // 256 * 256
    for B, T, H in [(16, 1024, 12), (2, 256, 3), (2, 37, 2), (1, 1, 1)]:
        small = lib.bt_attention_bwd_ws_min_bytes(B, T, H, 64)
        full = lib.bt_attention_bwd_ws_bytes(B, T, H, 64)
        assert small == al(4 * B * H * T)
        assert full == (small + al(4 * B * H * T * T) if T % 4 == 0 else small)
    assert lib.bt_attention_bwd_ws_bytes(0, 16, 1, 64) == 0
    # below the minimum workspace the call is rejected before any launch
    small = lib.bt_attention_bwd_ws_min_bytes(1, 16, 1, 64)
    assert lib.bt_attention_bwd(FAKE, FAKE + 8192, FAKE, FAKE, FAKE + 16384, FAKE + 32768, small - 1,
                                1, 16, 1, 64, None) == BT_EWORKSPACE


def test_cp_rank_segments_match_oracle_positions(lib):
    """The library's description of a rank's rows under the load-balanced
    split names the same global positions as the oracle's rearrangement."""
    from oracle import context_parallel as cp
    for T, W in [(256, 1), (1024, 2), (2048, 4), (16384, 8)]:
        for r in range(W):
            for s_ in (r, (r + 1) % W):
                g = bt.CPSegments()
                assert lib.bt_cp_rank_segments(T, W, r, s_, ctypes.byref(g)) == BT_OK
                assert g.seg == T // (2 * W) and g.n_q == 2 and g.n_k == 2

                def rows(pos):
                    return np.concatenate([np.arange(p, p + g.seg) for p in pos])
                assert np.array_equal(rows(g.q_pos), cp.rank_positions(T, W, r))
                assert np.array_equal(rows(g.k_pos), cp.rank_positions(T, W, s_))
    g = bt.CPSegments()
    assert lib.bt_cp_rank_segments(1000, 2, 0, 0, ctypes.byref(g)) == BT_ESHAPE
    assert lib.bt_cp_rank_segments(1024, 2, 2, 0, ctypes.byref(g)) == BT_EINVAL
    assert lib.bt_cp_rank_segments(1024, 2, 0, -1, ctypes.byref(g)) == BT_EINVAL
    assert lib.bt_cp_rank_segments(1024, 2, 0, 0, None) == BT_EINVAL
    assert lib.bt_cp_shard_tokens(FAKE, FAKE + 4096, 1, 1000, 2, 0, None) == BT_ESHAPE


def test_cp_block_validation(lib):
    def segs(seg=128, q=(0, 384), k=(128, 256)):
        return ctypes.byref(bt.cp_segments(seg, list(q), list(k)))
    H, hd = 2, 64
    fwd = lambda g, kvs=2 * H * hd, merge=0: lib.bt_attention_block_fwd(
        FAKE, FAKE + 65536, kvs, FAKE + 131072, FAKE + 196608, merge, 1, H, hd, g, None)
    assert fwd(segs(seg=100)) == BT_ESHAPE
    assert fwd(segs(seg=0)) == BT_ESHAPE
    assert fwd(segs(q=(0, 16))) == BT_ESHAPE             # position not a multiple of 32
    assert fwd(segs(k=(-128,))) == BT_ESHAPE
    g3 = bt.cp_segments(128, [0, 128], [0])
    g3.n_q = 3
    assert fwd(ctypes.byref(g3)) == BT_ESHAPE
    assert fwd(segs(), kvs=2 * H * hd - 4) == BT_ESHAPE  # K and V rows overlap
    assert fwd(segs(), kvs=2 * H * hd + 2) == BT_ESHAPE  # not a multiple of 4
    assert fwd(segs(), merge=2) == BT_EINVAL
    assert fwd(None) == BT_EINVAL
    assert lib.bt_attention_block_fwd(FAKE, FAKE_MIS, 2 * H * hd, FAKE + 131072, FAKE + 196608, 0, 1, H, hd,
                                      segs(), None) == BT_EALIGN
    bwd = lambda g, acc=0, dkv=FAKE + 262144, ws=None: lib.bt_attention_block_bwd(
        FAKE, FAKE + 65536, FAKE + 131072, 2 * H * hd, FAKE + 196608, FAKE + 200000, FAKE + 327680, dkv, acc,
        ws, 1 << 30, 1, H, hd, g, None)
    assert bwd(segs(), acc=4) == BT_EINVAL
    assert bwd(segs(), dkv=FAKE + 131072) == BT_EINVAL    # dkv aliases kv
    assert bwd(segs(seg=64)) == BT_ESHAPE
    assert bwd(segs(), ws=FAKE_MIS) == BT_EALIGN
    # stored-dS scratch: B H Tq Tk floats when every position is a multiple of 128, else none
    g = bt.cp_segments(256, [0, 512], [256, 768])
    assert lib.bt_attention_block_bwd_ws_bytes(2, 3, 64, ctypes.byref(g)) == 2 * 3 * 512 * 512 * 4
    g1 = bt.cp_segments(256, [0], [256, 768])
    assert lib.bt_attention_block_bwd_ws_bytes(1, 1, 64, ctypes.byref(g1)) == 256 * 512 * 4
    assert lib.bt_attention_block_bwd_ws_bytes(1, 1, 64, ctypes.byref(bt.cp_segments(256, [32], [0]))) == 0
    assert lib.bt_attention_block_bwd_ws_bytes(1, 1, 64, None) == 0
    assert lib.bt_attention_lse_merge(FAKE, FAKE, FAKE, FAKE, 1, 16, 2, 6, None) == BT_ESHAPE
    assert lib.bt_attention_lse_merge(FAKE, FAKE, None, FAKE, 1, 16, 2, 8, None) == BT_EINVAL
    assert lib.bt_attention_rowdot(FAKE, FAKE, FAKE, 1, 16, 2, 132, None) == BT_ESHAPE


def test_gpt2_context_validation(lib):
    cfg = bt.make_config(synth.TINY, synth.HP_TINY)
    need = lib.bt_gpt2_workspace_bytes(ctypes.byref(cfg), 2, 32)
    assert need > 0
    ctx = ctypes.c_void_p()
    assert lib.bt_gpt2_create(ctypes.byref(cfg), FAKE, need - 1, 2, 32, None, ctypes.byref(ctx)) == BT_EWORKSPACE
    assert lib.bt_gpt2_create(ctypes.byref(cfg), FAKE + 16, need, 2, 32, None, ctypes.byref(ctx)) == BT_EALIGN
    assert lib.bt_gpt2_create(ctypes.byref(cfg), FAKE, need, 2, 64, None, ctypes.byref(ctx)) == BT_ESHAPE
    bad = bt.make_config(synth.GPT2Config(V=10, Vp=12, max_T=8, L=1, H=1, C=256), synth.HP_TINY)
    assert lib.bt_gpt2_num_params(ctypes.byref(bad)) == 0  # head dim 256 unsupported
    assert lib.bt_gpt2_create(ctypes.byref(cfg), FAKE, need, 2, 32, None, ctypes.byref(ctx)) == BT_OK
    assert lib.bt_gpt2_step_count(ctx) == 0
    # a step larger than the context's token budget is rejected before any launch
    assert lib.bt_gpt2_fwd_bwd(ctx, FAKE, FAKE, FAKE, FAKE, 4, 32, 1.0, 0, None, None) == BT_ESHAPE
    # B*T not a multiple of 4 (the products need it): rejected before the embedding launches
    assert lib.bt_gpt2_fwd_bwd(ctx, FAKE, FAKE, FAKE, FAKE, 1, 31, 1.0, 0, None, None) == BT_ESHAPE
    assert b"multiple of 4" in lib.bt_last_error()
    lib.bt_gpt2_destroy(ctx)


def test_last_status_is_cleared_by_each_call(lib):
    assert lib.bt_gemm(0, 0, 5, 4, 4, FAKE, 4, FAKE, 4, 0.0, FAKE, 4, None, 0, None, None, None, None, None, 0,
                       None) == BT_ESHAPE
    assert lib.bt_last_status() == BT_ESHAPE and lib.bt_last_error() != b""
    # a later call that succeeds without launching anything clears both
    assert lib.bt_gelu_fwd(FAKE, FAKE, 0, None) == BT_OK
    assert lib.bt_last_status() == BT_OK and lib.bt_last_error() == b""
    assert lib.bt_embedding_index(FAKE, FAKE, 0, 2, 8, 100, None) == BT_EWORKSPACE
    assert lib.bt_last_status() == BT_EWORKSPACE
    assert lib.bt_embedding_bwd_indexed(FAKE, 1 << 20, FAKE, FAKE, FAKE, 0.5, FAKE, 1 << 20, 2, 8, 16, 100,
                                        None) == BT_EINVAL
