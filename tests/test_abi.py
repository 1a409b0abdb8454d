"""The C ABI library loads and exports every function include/lazytrain.h declares
(no compute calls: this runs without a GPU); the oracle library exports its own
header's functions.  Only host-side size queries are called."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header):
    with open(header) as fh:
        text = fh.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lto?_[a-z0-9_]+)\s*\(", text)))


def test_hip_library_exports_every_declared_symbol():
    import paper_2608_11919_amd as lt
    L = lt.lib()
    names = _declared(os.path.join(ROOT, "include", "lazytrain.h"))
    assert "lt_hybrid8bit_adamw_step" in names and "lt_grad_sqnorm" in names
    for n in names:
        assert hasattr(L, n), n


def test_oracle_library_exports_every_declared_symbol():
    import oracle
    L = oracle._load()
    for n in _declared(os.path.join(ROOT, "oracle", "lazytrain_oracle.h")):
        assert hasattr(L, n), n


def test_workspace_size_queries():
    import paper_2608_11919_amd as lt
    assert lt.lt_step_workspace_bytes(-1) == 0  # invalid
    assert lt.lt_step_workspace_bytes(0) > 0    # an empty list is valid: 0 means invalid
    assert lt.lt_step_workspace_bytes(325) >= 325 * 64
    assert lt.lt_grad_sqnorm_workspace_bytes([-1]) == 0
    assert lt.lt_grad_sqnorm_workspace_bytes([]) > 0
    assert lt.lt_grad_sqnorm_workspace_bytes([0, 0]) > 0
    assert lt.lib().lt_grad_sqnorm_workspace_bytes(None, 2) == 0  # numels NULL, n_tensors > 0
    small = lt.lt_grad_sqnorm_workspace_bytes([8192])
    big = lt.lt_grad_sqnorm_workspace_bytes([8192 * 1000 + 1])
    assert big - small >= 1000 * 8 - 256 and big % 256 == 0


def test_library_is_built_for_gfx950():
    so = os.path.join(ROOT, "paper_2608_11919_amd", "liblazytrain.so")
    with open(so, "rb") as fh:
        assert b"gfx950" in fh.read()


def test_product_path_never_imports_the_oracle():
    pkg = os.path.join(ROOT, "paper_2608_11919_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                with open(os.path.join(dirpath, f)) as fh:
                    src = fh.read()
                assert "import oracle" not in src and "lazytrain_oracle" not in src, f


def test_host_side_queries_of_the_next_rows():
    import paper_2608_11919_amd as lt
    assert lt.lt_grad_chunk_count([8192, 8193, 1]) == 4
    L = lt.lib()
    assert L.lt_grad_sqnorm_partials_workspace_bytes(-1) == 0
    assert L.lt_grad_sqnorm_partials_workspace_bytes(0) > 0
    assert L.lt_adamw_fp32_workspace_bytes(-1) == 0 and L.lt_adamw_fp32_workspace_bytes(0) > 0
    assert lt.lt_grad_chunk_count([0, 8193, 0]) == 2
    assert lt.lt_select_8bit_slice([], 0.5) == ([], 0)
    assert lt.lt_select_8bit_slice([0, 100, 0, 10], 0.1) == ([True, False, True, True], 10)
    assert L.lt_grad_sqnorm_partials_workspace_bytes(9) % 256 == 0
    assert L.lt_grad_sqnorm_finish_workspace_bytes(325) >= 326 * 8 + 325 * 8
    assert L.lt_adamw_fp32_workspace_bytes(4) >= 4 * 64
    numels, first = [4096, 300001, 9, 2048], [0, 2, 4]
    plain = lt.lt_streamed_workspace_bytes(numels, first, lt.LT_DTYPE_BF16, 2048, 3)
    copy = lt.lt_streamed_workspace_bytes(numels, first, lt.LT_DTYPE_BF16, 2048, 3, True)
    assert plain > 0 and copy > plain  # the bf16 copy needs room in every slot
    # resident gradients: the 3 slots (sized by layer 0) lose their gradient regions,
    # and every tensor gets one of its own, each rounded up to 256 bytes
    keep = lt.lt_streamed_workspace_bytes(numels, first, lt.LT_DTYPE_BF16, 2048, 3,
                                          keep_grads=True)
    up = lambda x: -(-x // 256) * 256
    assert keep == plain - 3 * (up(2 * 4096) + up(2 * 300001)) + sum(up(2 * n) for n in numels)
    assert lt.lt_streamed_workspace_bytes(numels, [0, 5], lt.LT_DTYPE_BF16, 2048, 3) == 0
    assert lt.lt_streamed_workspace_bytes(numels, first, lt.LT_DTYPE_BF16, 2048, 1) == 0


def test_streamed_optimizer_rejects_bad_arguments_before_any_device_work():
    import torch
    import paper_2608_11919_amd as lt
    w = [torch.zeros(4096), torch.zeros(10)]
    with pytest.raises(ValueError):
        lt.StreamedHybrid8bitAdamW([], [0], "cuda:0")
    with pytest.raises(ValueError):
        lt.StreamedHybrid8bitAdamW(w, [0, 2], "cuda:0", max_consecutive_skips=0)
    with pytest.raises(ValueError):
        lt.StreamedHybrid8bitAdamW(w, [0, 3], "cuda:0")  # layer_first past the list
    with pytest.raises(ValueError):
        lt.StreamedHybrid8bitAdamW(w, [0, 2], "cuda:0", ring_slots=1)
    with pytest.raises(ValueError):
        lt.StreamedHybrid8bitAdamW(w, [0, 2], "cuda:0", grad_dtype=torch.float16)
    with pytest.raises(TypeError):
        lt.StreamedHybrid8bitAdamW([torch.zeros(8, dtype=torch.float64)], [0, 1], "cuda:0")


def test_enum_values_match_the_binding():
    """The binding's constants are the header's values; the error codes are the
    boundary's (LT_ERR_HIP = 3, LT_ERR_WORKSPACE = 4)."""
    import paper_2608_11919_amd as lt
    with open(os.path.join(ROOT, "include", "lazytrain.h")) as fh:
        text = fh.read()
    names = ["LT_OK", "LT_ERR_INVALID_ARG", "LT_ERR_ALIGNMENT", "LT_ERR_HIP", "LT_ERR_WORKSPACE",
             "LT_STATUS_OK", "LT_STATUS_NONFINITE", "LT_STATUS_BAD_WORKSPACE", "LT_DTYPE_F32",
             "LT_DTYPE_BF16", "LT_MAP_LINEAR", "LT_MAP_DYNAMIC"]
    for name in names:
        m = re.search(rf"\b{name}\s*=\s*(\d+)", text)
        assert m, name
        assert int(m.group(1)) == getattr(lt, name), name
    assert (lt.LT_ERR_HIP, lt.LT_ERR_WORKSPACE) == (3, 4)


def test_hyperparameter_and_block_size_rejection_without_a_device():
    """Argument checks run before any pointer or device use, so they can be called
    here: eps must be positive also after rounding to fp32, block sizes are the
    multiples of 64 in [64, 65536]."""
    import paper_2608_11919_amd as lt
    L = lt.lib()
    # distinct fake device addresses (never dereferenced on these paths)
    one = lambda i: (ctypes.c_void_p * 1)(0x100000 * (i + 1))
    n1 = (ctypes.c_int64 * 1)(4096)

    def step(block, eps):
        return L.lt_hybrid8bit_adamw_step(one(0), one(1), lt.LT_DTYPE_BF16, one(2), one(3), one(4),
                                          one(5), None, n1, 1, block, lt.LT_MAP_LINEAR, 1e-4, 0.9,
                                          0.999, eps, 0.01, 1, None, None, None, None, 0, None)

    for eps in (0.0, -1e-8, 1e-50, float("inf"), float("nan")):
        assert step(2048, eps) == lt.LT_ERR_INVALID_ARG
        assert b"eps" in L.lt_last_error()
    for block in (0, 32, 1000, 65536 + 64, 1 << 20):
        assert step(block, 1e-8) == lt.LT_ERR_INVALID_ARG
        assert b"block_size" in L.lt_last_error()
    # valid values get past these checks (to the workspace check here: none is given)
    for block in (64, 192, 2048, 3072, 16384, 65536):
        assert step(block, 1e-8) == lt.LT_ERR_WORKSPACE
    assert L.lt_workspace_release(None) == lt.LT_OK
    assert L.lt_workspace_release(0x12345600) == lt.LT_OK  # unknown: a no-op
