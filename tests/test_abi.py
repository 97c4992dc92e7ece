"""CPU tests of the boundary: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before launching
anything (fake pointers below never reach a kernel)."""

import ctypes
import os
import re

import pytest

from tests._util import ROOT, ensure_built
from paper_2607_14107_amd import polestar as ps

INVALID, UNSUPPORTED, WORKSPACE = 1, 2, 4
FAKE = 0x10000          # 16-byte aligned, never dereferenced
MISALIGNED = 0x10004


@pytest.fixture(scope="module")
def L():
    return ensure_built()


def _header_functions():
    with open(os.path.join(ROOT, "include", "polestar.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(polestar_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = _header_functions()
    assert len(names) == 37, names
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings(L):
    assert L.polestar_version() == 10000
    for code in range(5):
        assert L.polestar_status_string(code)
    assert L.polestar_status_string(99) == b"unknown status"


def test_drift_validation(L):
    f = L.polestar_drift
    assert f(1, 1, 4, 8, None, FAKE, FAKE, None) == INVALID
    assert f(1, 0, 4, 8, FAKE, FAKE, FAKE, None) == INVALID
    assert f(2, 1, 4, 8, FAKE, FAKE, FAKE, None) == INVALID          # unknown dtype
    assert f(1, 1, 4, 12, FAKE, FAKE, FAKE, None) == UNSUPPORTED     # bf16 rows need d % 8 == 0
    assert f(0, 1, 4, 6, FAKE, FAKE, FAKE, None) == UNSUPPORTED      # fp32 rows need d % 4 == 0
    assert f(1, 1, 4, 8, MISALIGNED, FAKE, FAKE, None) == UNSUPPORTED
    assert f(1, 1, 4, 32768, FAKE, FAKE, FAKE, None) == UNSUPPORTED  # above the register budget


def test_select_validation(L):
    f = L.polestar_select
    assert f(1, 10, None, None, 0, 2, 3, FAKE, FAKE, None) == INVALID
    assert f(1, 10, FAKE, None, 0, 2, 11, FAKE, FAKE, None) == INVALID       # k > seq
    assert f(1, 10, FAKE, None, 9, 2, 3, FAKE, FAKE, None) == INVALID        # block past the end
    assert f(1, 10, FAKE, None, 0, 2, 3, None, FAKE, None) == INVALID        # k > 0 needs stale_idx
    assert f(1, 10, FAKE, None, -1, 2, 3, FAKE, FAKE, None) == INVALID
    assert f(1, 20000, FAKE, None, 0, 2, 3, FAKE, FAKE, None) == UNSUPPORTED


def test_refresh_noalloc_validation_and_limit(L):
    """The variant without a workspace validates like polestar_refresh_kv and
    refuses, before any GPU call, shapes whose scratch exceeds its array."""
    f = L.polestar_refresh_kv_noalloc
    limit = ps.refresh_kv_noalloc_max_bytes()
    assert limit == 64 << 20
    args = [1, 1, 768, 4096, 32, 128, FAKE, FAKE, FAKE, 115, 512, 32, FAKE, FAKE, FAKE, FAKE, None]
    a = list(args); a[6] = None
    assert f(*a) == INVALID                                   # h_cur
    a = list(args); a[10] = 760
    assert f(*a) == INVALID                                   # block past the end
    a = list(args); a[7] = None
    assert f(*a) == INVALID                                   # k_max > 0 needs stale_idx
    a = list(args); a[5] = 96
    assert f(*a) == UNSUPPORTED                               # head_dim
    a = list(args); a[15] = MISALIGNED
    assert f(*a) == UNSUPPORTED
    # 8 sequences x (100 stale + 32 block rows) onto 64 x 128 K and V columns
    # from d = 8192: the plan splits K, 132 MiB of partials
    assert ps.refresh_kv_workspace_size(ps.BF16, 8, 8192, 64, 128, 100, 32) > limit
    big = [1, 8, 160, 8192, 64, 128, FAKE, FAKE, FAKE, 100, 128, 32, FAKE, FAKE, FAKE, FAKE, None]
    assert f(*big) == WORKSPACE


def test_refresh_validation_and_workspace(L):
    f = L.polestar_refresh_kv
    ws = ps.refresh_kv_workspace_size(ps.BF16, 1, 4096, 32, 128, 115, 32)
    assert ws > 0
    args = [1, 1, 768, 4096, 32, 128, FAKE, FAKE, FAKE, 115, 512, 32, FAKE, FAKE, FAKE, FAKE, FAKE, ws, None]
    a = list(args); a[6] = None
    assert f(*a) == INVALID                                   # h_cur
    a = list(args); a[10] = 760
    assert f(*a) == INVALID                                   # block past the end
    a = list(args); a[7] = None
    assert f(*a) == INVALID                                   # k_max > 0 needs stale_idx
    a = list(args); a[5] = 96
    assert f(*a) == UNSUPPORTED                               # head_dim
    a = list(args); a[14] = MISALIGNED
    assert f(*a) == UNSUPPORTED
    a = list(args); a[17] = ws - 1
    assert f(*a) == WORKSPACE
    # nothing to refresh: returns OK without launching
    a = list(args); a[9] = 0; a[11] = 0; a[7] = None; a[8] = None
    assert f(*a) == 0
    assert ps.refresh_kv_workspace_size(ps.BF16, 1, 4096, 32, 128, -1, 32) == 0


def test_attend_validation_and_workspace(L):
    f = L.polestar_attend
    ws = ps.attend_workspace_size(ps.BF16, 1, 768, 4096, 32, 32, 128, 32)
    assert ws > 0
    args = [1, 1, 768, 4096, 32, 32, 128, 512, 32, FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, None, FAKE, ws, None]
    a = list(args); a[5] = 5
    assert f(*a) == INVALID                                   # heads % kv_heads
    a = list(args); a[8] = 0
    assert f(*a) == INVALID                                   # empty block
    a = list(args); a[9] = None
    assert f(*a) == INVALID                                   # w_q without h_cur
    a = list(args); a[6] = 256
    assert f(*a) == UNSUPPORTED
    a = list(args); a[18] = ws - 1
    assert f(*a) == WORKSPACE


def test_project_q_validation_and_workspace(L):
    f = L.polestar_project_q
    assert ps.project_q_workspace_size(ps.BF16, 1, 4096, 32, 128, 16) == 0      # 16 rows: small kernel, no partials
    assert ps.project_q_workspace_size(ps.FP32, 1, 4096, 32, 128, 32) == 0      # fp32: small kernel
    assert ps.project_q_workspace_size(ps.BF16, 1, 4096, 32, 128, 32) > 0       # 32 bf16 rows: DMA kernel, split-K
    ws = ps.project_q_workspace_size(ps.BF16, 8, 4096, 32, 128, 32)
    assert ws > 0                                                                # 256 rows: split-K
    args = [1, 8, 1536, 4096, 32, 128, 1024, 32, FAKE, FAKE, FAKE, FAKE, ws, None]
    a = list(args); a[8] = None
    assert f(*a) == INVALID                                   # h_cur
    a = list(args); a[6] = 1510
    assert f(*a) == INVALID                                   # block past the end
    a = list(args); a[7] = 0
    assert f(*a) == INVALID                                   # empty block
    a = list(args); a[3] = 4000
    assert f(*a) == UNSUPPORTED                               # d % 128
    a = list(args); a[5] = 96
    assert f(*a) == UNSUPPORTED                               # head_dim
    a = list(args); a[10] = MISALIGNED
    assert f(*a) == UNSUPPORTED
    a = list(args); a[12] = ws - 1
    assert f(*a) == WORKSPACE


def test_commit_validation_and_workspace(L):
    f = L.polestar_commit
    ws = ps.commit_workspace_size(ps.BF16, 1, 32, 126464)
    assert ws > 0
    args = [1, 1, 32, 126464, FAKE, FAKE, FAKE, 768, 512, FAKE, FAKE, 5, -1, 0.9, 10.0, 1,
            FAKE, FAKE, FAKE, FAKE, ws, None]
    a = list(args); a[4] = None
    assert f(*a) == INVALID
    a = list(args); a[12] = 126464
    assert f(*a) == INVALID                                   # mask id beyond the vocabulary
    a = list(args); a[9] = None
    assert f(*a) == INVALID                                   # h > 0 with drift needs hist
    a = list(args); a[8] = 740
    assert f(*a) == INVALID                                   # block past the end of drift rows
    a = list(args); a[3] = 126465
    assert f(*a) == UNSUPPORTED                               # rows of 16-byte chunks
    a = list(args); a[20] = ws - 1
    assert f(*a) == WORKSPACE


def test_suffix_commit_validation(L):
    f = L.polestar_suffix_commit
    ws = ps.commit_workspace_size(ps.BF16, 1, 32, 126464)
    args = [1, 1, 32, 126464, FAKE, FAKE, FAKE, -1, 0.9, FAKE, FAKE, FAKE, FAKE, ws, None]
    a = list(args); a[6] = None
    assert f(*a) == INVALID                                   # eligibility mask required
    a = list(args); a[7] = 126464
    assert f(*a) == INVALID
    a = list(args); a[2] = 1025
    assert f(*a) == UNSUPPORTED
    a = list(args); a[3] = 126465
    assert f(*a) == UNSUPPORTED
    a = list(args); a[13] = ws - 1
    assert f(*a) == WORKSPACE


def test_model_entry_validation(L):
    # embed: rows past the sequence, width not a multiple of 4
    assert L.polestar_embed(1, 2, 96, 256, FAKE, 90, 10, FAKE, 512, FAKE, FAKE, None) == INVALID
    assert L.polestar_embed(1, 2, 96, 254, FAKE, 0, 10, FAKE, 512, FAKE, FAKE, None) == UNSUPPORTED
    assert L.polestar_embed(1, 2, 96, 256, FAKE, 0, 10, FAKE, 512, FAKE, MISALIGNED, None) == UNSUPPORTED
    # rmsnorm: destination rows past its sequence, negative eps, width too large
    assert L.polestar_rmsnorm(1, 2, 10, 256, FAKE, 10, 0, 1e-5, FAKE, 12, 3, None) == INVALID
    assert L.polestar_rmsnorm(1, 2, 10, 256, FAKE, 10, 0, -1.0, FAKE, 12, 0, None) == INVALID
    assert L.polestar_rmsnorm(1, 2, 10, 16388, FAKE, 10, 0, 1e-5, FAKE, 12, 0, None) == UNSUPPORTED
    # linear: K not a multiple of 128 (bf16), N not of 16, workspace
    assert L.polestar_linear(1, 2, 50, 384, 272, 45, 10, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == INVALID
    assert L.polestar_linear(1, 2, 50, 320, 272, 0, 10, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == UNSUPPORTED
    assert L.polestar_linear(1, 2, 50, 384, 270, 0, 10, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == UNSUPPORTED
    ws = ps.linear_workspace_size(ps.BF16, 2, 200, 256, 4096)
    assert ws > 0
    assert L.polestar_linear(1, 2, 200, 4096, 256, 0, 200, FAKE, FAKE, FAKE, FAKE, ws - 1, None) == WORKSPACE
    # swiglu / residual add / copy rows
    assert L.polestar_swiglu(1, 10, 6, FAKE, FAKE, None) == UNSUPPORTED
    assert L.polestar_swiglu(1, 10, 8, None, FAKE, None) == INVALID
    assert L.polestar_residual_add(1, 10, FAKE, FAKE, None) == UNSUPPORTED
    assert L.polestar_residual_add(1, 0, None, None, None) == 0           # nothing to do
    assert L.polestar_copy_rows(1, 2, 96, 256, FAKE, FAKE, None, None, 4, 0, 32, None) == INVALID
    assert L.polestar_copy_rows(1, 2, 96, 4, FAKE, FAKE, None, None, 0, 0, 32, None) == UNSUPPORTED
    assert L.polestar_copy_rows(1, 2, 96, 256, FAKE, FAKE, None, None, 0, 80, 32, None) == INVALID
    for f in (L.polestar_gather_rows, L.polestar_scatter_rows):
        assert f(2, 96, 512, FAKE, None, FAKE, 8, FAKE, None) == INVALID     # rows need indices
        assert f(2, 96, 500, FAKE, FAKE, FAKE, 8, FAKE, None) == UNSUPPORTED
        assert f(2, 96, 512, FAKE, FAKE, FAKE, 8, MISALIGNED, None) == UNSUPPORTED
        assert f(2, 96, 512, None, None, None, 0, None, None) == 0          # nothing to move
    # codec
    assert L.polestar_codec_row_bytes(0, 4096) == 2048 and L.polestar_codec_row_bytes(1, 4096) == 4096
    assert L.polestar_codec_row_bytes(2, 4096) == 0 and L.polestar_codec_row_bytes(0, 4010) == 0
    assert L.polestar_cluster_means(2, 96, 512, FAKE, FAKE, 32, FAKE, 17, FAKE, None) == UNSUPPORTED
    assert L.polestar_cluster_means(2, 96, 512, None, FAKE, 32, FAKE, 8, FAKE, None) == INVALID
    enc = L.polestar_codec_encode
    assert enc(2, 2, 96, 512, FAKE, FAKE, FAKE, 8, FAKE, 8, FAKE, FAKE, FAKE, None) == INVALID     # format
    assert enc(0, 2, 96, 500, FAKE, FAKE, FAKE, 8, FAKE, 8, FAKE, FAKE, FAKE, None) == UNSUPPORTED
    assert enc(0, 2, 96, 512, FAKE, None, FAKE, 8, FAKE, 8, FAKE, FAKE, FAKE, None) == INVALID
    gat = L.polestar_codec_gather
    assert gat(0, 1, 2, 96, 512, FAKE, FAKE, FAKE, FAKE, 8, FAKE, 8, FAKE, -1.0, FAKE, None, None) == INVALID
    assert gat(0, 1, 2, 96, 512, FAKE, FAKE, FAKE, FAKE, 8, FAKE, 8, FAKE, 1e-5, MISALIGNED, None, None) == UNSUPPORTED


def test_attention_drift_validation(L):
    f = L.polestar_attention_drift
    ws = ps.attention_drift_workspace_size(1, 768, 32, 32)
    assert ws > 0
    args = [1, 1, 768, 32, 32, 32, 128, FAKE, FAKE, 0.0, FAKE, FAKE, 0, FAKE, FAKE, ws, None]
    a = list(args); a[12 + 1] = None
    assert f(*a) == INVALID                                   # drift output required
    a = list(args); a[5] = 5
    assert f(*a) == INVALID                                   # heads not a multiple of kv heads
    a = list(args); a[3] = 65
    assert f(*a) == UNSUPPORTED                               # more than 64 query rows
    a = list(args); a[6] = 96
    assert f(*a) == UNSUPPORTED
    a = list(args); a[7] = MISALIGNED
    assert f(*a) == UNSUPPORTED
    a = list(args); a[15] = ws - 1
    assert f(*a) == WORKSPACE


def test_step_validation_and_workspace(L):
    a = ps.StepArgs()
    a.dtype, a.batch, a.seq, a.d = 1, 1, 768, 4096
    a.n_heads, a.n_kv_heads, a.head_dim = 32, 32, 128
    a.block_start, a.block_len, a.vocab, a.k, a.h = 512, 32, 126464, 106, 5
    a.mask_token_id, a.tau_s, a.alpha = -1, 0.9, 10.0
    ws = ps.step_workspace_size(a)
    assert ws > 0
    # sum of the pieces' workspaces (refresh, attention partials, scan partials)
    parts = (ps.refresh_kv_workspace_size(1, 1, 4096, 32, 128, 106, 32)
             + ps.attend_workspace_size(1, 1, 768, 4096, 32, 32, 128, 32)
             + ps.commit_workspace_size(1, 1, 32, 126464))
    assert parts <= ws <= parts + 4 * 256
    f = L.polestar_step
    assert f(ctypes.byref(a), FAKE, ws, None, None, None) == INVALID      # pointers missing
    for name in ("h_cur", "h_prev", "w_q", "w_k", "w_v", "k_cache", "v_cache", "logits", "masked", "hist",
                 "hist_len", "drift", "stale_idx", "stale_count", "q", "out", "token", "conf", "commit"):
        setattr(a, name, FAKE)
    assert f(ctypes.byref(a), FAKE, ws - 1, None, None, None) == WORKSPACE
    a.block_start = 740
    assert f(ctypes.byref(a), FAKE, ws, None, None, None) == INVALID      # block past the end
    a.block_start = 512
    a.n_kv_heads = 5
    assert f(ctypes.byref(a), FAKE, 1 << 30, None, None, None) == INVALID  # heads % kv heads
    a.n_kv_heads = 32
    a.h_cur = MISALIGNED
    assert f(ctypes.byref(a), FAKE, ws, None, None, None) == UNSUPPORTED
    assert L.polestar_step(None, FAKE, ws, None, None, None) == INVALID
    assert L.polestar_step_workspace_size(None) == 0


def test_proxy_calls_validation(L):
    c = L.polestar_cluster
    args = [1, 1, 768, 4096, FAKE, FAKE, 96, 8, 10, FAKE, FAKE, FAKE, FAKE, None]
    a = list(args); a[4] = None
    assert c(*a) == INVALID
    a = list(args); a[7] = 97
    assert c(*a) == INVALID                                   # more clusters than points
    a = list(args); a[7] = 17
    a[6] = 200
    assert c(*a) == UNSUPPORTED                               # K above 16
    a = list(args); a[3] = 8192
    assert c(*a) == UNSUPPORTED                               # K * d above the LDS budget
    ws = ps.proxy_drift_workspace_size(1, 1, 768, 4096, 32, 128, 8)
    assert ws > 0
    f = L.polestar_proxy_drift
    pa = [1, 1, 768, 4096, 32, 32, 128, 8, FAKE, FAKE, FAKE, FAKE, 0.0, FAKE, FAKE, 0, FAKE, FAKE, ws, None]
    a = list(pa); a[5] = 5
    assert f(*a) == INVALID                                   # heads % kv heads
    a = list(pa); a[6] = 96
    assert f(*a) == UNSUPPORTED
    a = list(pa); a[18] = ws - 1
    assert f(*a) == WORKSPACE
    s = L.polestar_cluster_select
    assert s(1, 768, FAKE, 8, FAKE, 4, None, 10, FAKE, None) == INVALID        # k_max > 0 needs stale_idx
    assert s(1, 768, FAKE, 17, FAKE, 4, FAKE, 10, FAKE, None) == UNSUPPORTED
    u = L.polestar_cluster_update
    assert u(1, 1, 768, 4096, FAKE, FAKE, FAKE, 8, FAKE, FAKE, 10, None, None) == INVALID   # sums
    assert u(1, 1, 768, 4094, FAKE, FAKE, FAKE, 8, FAKE, FAKE, 10, FAKE, None) == UNSUPPORTED
    assert u(1, 1, 768, 4096, FAKE, FAKE, FAKE, 8, FAKE, FAKE, 0, FAKE, None) == 0         # nothing refreshed


def test_binding_fails_loudly_without_gpu_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 4, 8)
    with pytest.raises(ValueError):
        ps.drift(x, x)
