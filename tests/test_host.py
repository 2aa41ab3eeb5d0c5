"""Host-side logic that needs no GPU: the C ABI loads and exports what the
header declares, argument checks fail before any launch, workspace sizing,
and the algorithmic work counters against closed forms and the paper's
figures."""
import ctypes
import json
import os

import numpy as np
import pytest

import paper_2608_23658_amd.kvattn as K
from paper_2608_23658_amd import work

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def L():
    return K.lib()


def test_library_exports_every_declared_symbol(L):
    names = K.declared_symbols()
    assert len(names) >= 16
    for n in names:
        assert hasattr(L, n), n
    assert L.kvattn_abi_version() == 1


# fake, 16-byte-aligned non-null addresses: every call below must be rejected
# by the host checks, before anything is launched
A = 1 << 20


def _decode(L, **kw):
    a = dict(q=A, kv=A, nb=100, bt=A, sl=A, out=A, B=4, hq=32, hkv=8, d=128, bs=16, mb=10,
             msl=160, scale=0.1, dt=K.KV_BF16, ws=A, wsb=1 << 30, stream=None)
    a.update(kw)
    return L.kvattn_decode(a["q"], a["kv"], a["nb"], a["bt"], a["sl"], a["out"], a["B"], a["hq"],
                           a["hkv"], a["d"], a["bs"], a["mb"], a["msl"], a["scale"], a["dt"],
                           a["ws"], a["wsb"], a["stream"])


def _prefill(L, **kw):
    a = dict(q=A, kv=A, nb=100, bt=A, sl=A, cu=A, out=A, B=2, T=100, budget=128, hq=32, hkv=8,
             d=128, bs=16, mb=10, msl=160, scale=0.1, dt=K.KV_BF16, ws=A, wsb=1 << 20,
             stream=None)
    a.update(kw)
    return L.kvattn_prefill_chunk(a["q"], a["kv"], a["nb"], a["bt"], a["sl"], a["cu"], a["out"],
                                  a["B"], a["T"], a["budget"], a["hq"], a["hkv"], a["d"], a["bs"],
                                  a["mb"], a["msl"], a["scale"], a["dt"], a["ws"], a["wsb"],
                                  a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(d=96), K.KV_ERR_UNSUPPORTED),
    (dict(d=128, dt=K.KV_F32), K.KV_ERR_UNSUPPORTED),
    (dict(hq=24, hkv=8), K.KV_ERR_UNSUPPORTED),          # group of 3
    (dict(hq=30, hkv=8), K.KV_ERR_INVALID),
    (dict(bs=32), K.KV_ERR_UNSUPPORTED),
    (dict(dt=7), K.KV_ERR_INVALID),
    (dict(msl=161), K.KV_ERR_INVALID),                   # > max_blocks * block_size
    (dict(nb=0), K.KV_ERR_INVALID),
    (dict(q=A + 8), K.KV_ERR_INVALID),                   # misaligned
    (dict(out=0), K.KV_ERR_INVALID),
    (dict(wsb=100), K.KV_ERR_INVALID),                   # workspace too small
    (dict(scale=float("inf")), K.KV_ERR_INVALID),
    (dict(B=-1), K.KV_ERR_INVALID),
])
def test_decode_argument_checks(L, kw, code):
    assert _decode(L, **kw) == code
    assert K.last_error().startswith("kvattn_decode")


def _decode2(L, **kw):
    a = dict(q=A, kb=A, nbase=80, ke=A, nel=20, bt=A, sl=A, out=A, B=4, hq=32, hkv=8, d=128,
             bs=16, mb=10, msl=160, scale=0.1, dt=K.KV_BF16, ws=A, wsb=1 << 30, stream=None)
    a.update(kw)
    return L.kvattn_decode_two_tensor(a["q"], a["kb"], a["nbase"], a["ke"], a["nel"], a["bt"],
                                      a["sl"], a["out"], a["B"], a["hq"], a["hkv"], a["d"],
                                      a["bs"], a["mb"], a["msl"], a["scale"], a["dt"], a["ws"],
                                      a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dt=K.KV_F32, d=64), K.KV_ERR_UNSUPPORTED),
    (dict(d=64), K.KV_ERR_UNSUPPORTED),
    (dict(nel=0), K.KV_ERR_INVALID),
    (dict(nbase=0), K.KV_ERR_INVALID),
    (dict(ke=A + 8), K.KV_ERR_INVALID),
    (dict(ke=0), K.KV_ERR_INVALID),
    (dict(wsb=100), K.KV_ERR_INVALID),
    (dict(bs=32), K.KV_ERR_UNSUPPORTED),
])
def test_decode_two_tensor_argument_checks(L, kw, code):
    assert _decode2(L, **kw) == code
    assert K.last_error().startswith("kvattn_decode_two_tensor")


def test_decode_empty_batch_is_ok(L):
    assert _decode(L, B=0, q=0, out=0) == K.KV_OK
    assert K.last_error() == ""


@pytest.mark.parametrize("kw,code", [
    (dict(dt=K.KV_F32), K.KV_ERR_UNSUPPORTED),
    (dict(d=64), K.KV_ERR_UNSUPPORTED),
    (dict(hq=128, hkv=8), K.KV_ERR_UNSUPPORTED),         # group of 16 is not built
    (dict(T=200, budget=128), K.KV_ERR_INVALID),         # over max_num_batched_tokens
    (dict(cu=0), K.KV_ERR_INVALID),
    (dict(wsb=16), K.KV_ERR_INVALID),
    (dict(msl=1000), K.KV_ERR_INVALID),
])
def test_prefill_argument_checks(L, kw, code):
    assert _prefill(L, **kw) == code


def _append(L, **kw):
    a = dict(k=A, v=A, sm=A, kv=A, nb=100, T=64, hkv=8, d=128, bs=16, dt=K.KV_BF16,
             stream=None)
    a.update(kw)
    return L.kvattn_kv_append(a["k"], a["v"], a["sm"], a["kv"], a["nb"], a["T"], a["hkv"],
                              a["d"], a["bs"], a["dt"], a["stream"])


@pytest.mark.parametrize("kw,code", [
    (dict(dt=5), K.KV_ERR_INVALID),
    (dict(T=-1), K.KV_ERR_INVALID),
    (dict(d=12), K.KV_ERR_INVALID),                      # 24-byte rows: not whole chunks
    (dict(d=4, dt=K.KV_BF16), K.KV_ERR_INVALID),
    (dict(d=8), K.KV_ERR_UNSUPPORTED),                   # 16-byte rows
    (dict(d=320), K.KV_ERR_UNSUPPORTED),                 # 640-byte rows
    (dict(hkv=0), K.KV_ERR_INVALID),
    (dict(bs=32), K.KV_ERR_UNSUPPORTED),
    (dict(nb=0), K.KV_ERR_INVALID),
    (dict(nb=1 << 28), K.KV_ERR_INVALID),                # slots overflow int32
    (dict(sm=0), K.KV_ERR_INVALID),
    (dict(k=A + 4), K.KV_ERR_INVALID),                   # misaligned
])
def test_append_argument_checks(L, kw, code):
    assert _append(L, **kw) == code
    assert K.last_error().startswith("kvattn_kv_append")


def test_append_nothing_is_ok(L):
    assert _append(L, T=0, k=0, v=0, sm=0) == K.KV_OK


def test_workspace_sizes():
    split = K.decode_split_tokens(4096)
    assert split % 64 == 0 and split > 0
    need = K.decode_workspace_bytes(256, 32, 128, 4096)
    splits = -(-4096 // split)
    assert need >= 256 * 32 * splits * (128 + 2) * 4
    assert K.decode_workspace_bytes(-1, 32, 128, 4096) == 0
    assert K.prefill_workspace_bytes(129, 8320, 32, 128) >= (8320 // 64 + 129) * 8


def test_pool_rejects_bad_sizes_without_a_device(L):
    h = ctypes.c_void_p()
    assert L.kvpool_create(0, 0, 1 << 21, 1 << 21, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert L.kvpool_create(0, 2, 0, 0, ctypes.byref(h)) == K.KV_ERR_INVALID
    assert not h.value
    assert L.kvpool_commit_elastic(None, None) == K.KV_ERR_INVALID
    assert L.kvpool_decommit_elastic(None, None) == K.KV_ERR_INVALID
    assert L.kvpool_is_committed(None) == K.KV_ERR_INVALID
    L.kvpool_destroy(None)


def test_prefill_pairs_closed_forms_and_chunk_identity():
    Lt = 32768
    whole = work.prefill_pairs([Lt], [Lt])
    assert whole == Lt * (Lt + 1) // 2 == 536_887_296
    parts = [work.prefill_pairs([8192 * (k + 1)], [8192]) for k in range(4)]
    assert sum(parts) == whole
    assert parts == [33_558_528, 100_667_392, 167_776_256, 234_885_120]
    # brute-force count on a small case
    for L_, n in [(37, 37), (100, 20), (300, 1), (513, 257)]:
        c = L_ - n
        brute = sum(1 for i in range(n) for t in range(L_) if t <= c + i)
        assert work.prefill_pairs([L_], [n]) == brute


def test_flop_and_byte_counts():
    # the last 8192-token chunk of a 32768-token prompt at 32 heads of 128
    assert work.prefill_flops([32768], [8192], 32, 128) == 16384 * 234_885_120   # 3.848 TFLOP
    assert work.prefill_flops([32768], [32768], 32, 128) == 4 * 128 * 32 * 536_887_296
    # 4096 bytes of K+V per token per layer at 8 kv heads of 128 in bf16
    assert work.decode_kv_bytes([1, 2, 3], 8, 128, 2) == 6 * 4096
    b = work.decode_bytes([16, 17], 32, 8, 128, 2)
    assert b == 33 * 4096 + 2 * 2 * 32 * 128 * 2 + 3 * 4 + 8


def test_paper_figures_fixture():
    """Figures the paper prints that bound the workloads (see the fixture's
    citations): the decode share of the chunk budget and the toggle reserve."""
    with open(os.path.join(GOLDEN, "paper_figures.json")) as f:
        fig = json.load(f)
    share = fig["decode_tokens_at_max_batch"] / fig["chunk_budget_small"]
    assert abs(share - fig["decode_share_of_budget"]) < 0.005
    # the 3 GiB reserve in 2 MiB granules spreads over 28 layers at ~56 granules each
    per_layer = fig["reserve_gib"] * 1024 / fig["num_layers"]
    assert 55 <= per_layer / fig["vmm_granularity_mib"] <= 57
    assert fig["chunk_budget_large"] // fig["chunk_budget_small"] == 4


def test_c_client_builds_against_the_header_and_runs(tmp_path):
    """The header is plain C99 and the library links and works from C: a small
    client (tests/c_abi_client.c) compiled with gcc -std=c99 -pedantic -Werror
    against include/kvattn.h and the built library makes the GPU-free calls."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    K.lib()   # the library must be built
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.dirname(K.LIB_PATH)
    exe = str(tmp_path / "c_abi_client")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "c_abi_client.c"),
                    "-L", libdir, "-l:libkvattn.so", "-Wl,-rpath," + libdir, "-o", exe],
                   check=True, capture_output=True, text=True)
    env = dict(os.environ)
    env["LD_LIBRARY_PATH"] = os.pathsep.join(
        [p for p in ("/opt/rocm/lib", env.get("LD_LIBRARY_PATH", "")) if p])
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("ALL OK"), r.stdout


def test_block_pool_and_controller_under_sanitizers(tmp_path):
    """The block-id pool and the toggle controller (csrc/blockpool.cpp, host
    code) built with g++ and the address and undefined-behaviour sanitizers,
    driven by tests/host_fuzz.cpp: 20000 random allocations, frees, bad frees,
    drains and scheduler steps per seed against a plain model, with the pool's
    commit and decommit failing now and then the ways the real pool can."""
    import shutil
    import subprocess
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = str(tmp_path / "host_fuzz")
    r = subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                        "-I", os.path.join(root, "include"),
                        "-I", os.path.join(root, "paper_2608_23658_amd", "csrc"),
                        os.path.join(root, "tests", "host_fuzz.cpp"),
                        os.path.join(root, "paper_2608_23658_amd", "csrc", "blockpool.cpp"),
                        "-o", exe], capture_output=True, text=True)
    if r.returncode != 0 and "sanitizer" in (r.stderr or "").lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr
    for seed in (7, 8, 9):
        r = subprocess.run([exe, "20000", str(seed)], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0, (seed, r.stdout + r.stderr)
        assert r.stdout.startswith("ok:"), r.stdout


def test_binding_rejects_views_and_wide_indices_before_any_launch():
    """Tensors reach the library as bare pointers: a strided view or an int64
    index tensor is refused by the binding, before the library is called."""
    import torch
    q = torch.zeros(4, 8, 128, dtype=torch.bfloat16)
    bt = torch.zeros(4, 3, dtype=torch.int32)
    sl = torch.ones(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="int32"):
        K.decode(q, 0, 10, bt.long(), sl, num_kv_heads=2, max_seq_len=48)
    strided = torch.zeros(4, 8, 256, dtype=torch.bfloat16)[:, :, :128]
    with pytest.raises(ValueError, match="contiguous"):
        K.decode(strided, 0, 10, bt, sl, num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="block_table"):
        K.decode(q, 0, 10, bt.flatten(), sl, num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="out"):
        K.decode(q, 0, 10, bt, sl, num_kv_heads=2, max_seq_len=48, out=q.float())
    cu = torch.tensor([0, 1, 2, 3, 4], dtype=torch.int64)
    with pytest.raises(ValueError, match="cu_seqlens_q"):
        K.prefill_chunk(q, 0, 10, bt, sl, cu, num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="GPU"):
        K.decode(q, 0, 10, bt, sl, num_kv_heads=2, max_seq_len=48)


def test_binding_checks_batch_lengths_before_any_launch():
    """seq_lens, the block-table rows and cu_seqlens_q reach the kernels as
    bare pointers indexed by sequence: lengths that do not match the batch
    would make them read past the tensors, so the binding refuses them."""
    import torch
    q = torch.zeros(4, 8, 128, dtype=torch.bfloat16)
    bt = torch.zeros(4, 3, dtype=torch.int32)
    sl = torch.ones(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="seq_lens"):
        K.decode(q, 0, 10, bt, sl[:3], num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="block_table"):
        K.decode(q, 0, 10, bt[:3], sl, num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="seq_lens"):
        K.decode_two_tensor(q, 0, 5, 0, 5, bt, sl[:2], num_kv_heads=2, max_seq_len=48)
    out = torch.empty_like(q)
    with pytest.raises(ValueError, match="block_table"):
        K.decode_noalloc(q, 0, 10, bt[:2], sl, out, num_kv_heads=2, max_seq_len=48)
    # prefill: 2 sequences over 4 new rows
    cu = torch.tensor([0, 2, 4], dtype=torch.int32)
    with pytest.raises(ValueError, match="cu_seqlens_q"):
        K.prefill_chunk(q, 0, 10, bt[:2], sl[:2], cu[:2], num_kv_heads=2, max_seq_len=48)
    with pytest.raises(ValueError, match="block_table"):
        K.prefill_chunk(q, 0, 10, bt, sl[:2], cu, num_kv_heads=2, max_seq_len=48)


def test_noalloc_decode_refuses_before_touching_a_device(L):
    """The allocation-free decode checks its sizes against its static scratch
    (and the rest of its arguments) on the host, before any HIP call."""
    cap = L.kvattn_decode_noalloc_max_scratch_bytes()
    assert cap == 32 << 20

    def call(**kw):
        a = dict(B=256, hq=32, hkv=8, d=128, mb=4096, msl=4096 * 16, dt=K.KV_BF16)
        a.update(kw)
        return L.kvattn_decode_noalloc(A, A, 100, A, A, A, a["B"], a["hq"], a["hkv"], a["d"], 16,
                                       a["mb"], a["msl"], 0.1, a["dt"], None)
    assert call() == K.KV_ERR_INVALID                   # 64 splits of 256 x 32 rows: too big
    assert "static scratch" in K.last_error()
    assert K.decode_workspace_bytes(256, 32, 128, 4096 * 16) > cap
    assert call(d=96, msl=160, mb=10) == K.KV_ERR_UNSUPPORTED
    assert call(hq=30, msl=160, mb=10) == K.KV_ERR_INVALID
    assert call(B=-1) == K.KV_ERR_INVALID
    assert call(B=0, msl=160, mb=10) == K.KV_OK          # nothing to do


def test_probes_refuse_bad_arguments_before_any_launch(L):
    """The rate probes check their arguments on the host; none of these
    calls reaches a device."""
    assert L.kvattn_probe_mfma_threads() == 512
    assert L.kvattn_probe_mfma(None, None, 1, 1, None) == K.KV_ERR_INVALID
    assert L.kvattn_probe_mfma(A, None, 0, 1, None) == K.KV_ERR_INVALID
    assert L.kvattn_probe_mfma(A, A, 1, -1, None) == K.KV_ERR_INVALID
    assert L.kvattn_probe_read_blocks_waves(256, 8, 4096) == 256 * 8 * 4
    assert L.kvattn_probe_read_blocks_waves(256, 8, 4097) == 256 * 8 * 5
    assert L.kvattn_probe_read_blocks_waves(0, 8, 4096) == 0
    assert L.kvattn_probe_read_blocks_waves(1 << 20, 64, 1 << 20) == -1

    def read(**kw):
        a = dict(kv=A, nb=10, bt=A, sl=A, B=4, hkv=8, d=128, dt=K.KV_BF16, mb=10, msl=160,
                 out=A)
        a.update(kw)
        return L.kvattn_probe_read_blocks(a["kv"], a["nb"], a["bt"], a["sl"], a["B"], a["hkv"],
                                          a["d"], a["dt"], a["mb"], a["msl"], a["out"], None)
    assert read(d=16) == K.KV_ERR_UNSUPPORTED      # a 512-byte tile
    assert read(d=64) == K.KV_ERR_UNSUPPORTED      # bf16 with head_dim 64: 2 KiB tiles
    assert read(dt=7) == K.KV_ERR_INVALID
    assert read(kv=A + 8) == K.KV_ERR_INVALID       # not 16-byte aligned
    assert read(bt=None) == K.KV_ERR_INVALID
    assert read(out=None) == K.KV_ERR_INVALID
    assert read(B=0) == K.KV_ERR_INVALID
    assert read(nb=0) == K.KV_ERR_INVALID
