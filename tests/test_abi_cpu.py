"""The C ABI on the host: every symbol include/zo.h declares is exported, and
argument errors are reported before anything is launched (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2608_15665_amd as zo
from paper_2608_15665_amd._lib import Panel, UpdateItem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "zo.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(zo_\w+)\s*\(", src)))


def test_header_declares_the_abi():
    fns = header_functions()
    assert set(fns) == set(zo.ABI_SYMBOLS), fns


def test_library_exports_every_declared_symbol():
    L = zo.lib()
    for name in header_functions():
        assert hasattr(L, name), name
    assert zo.abi_version() == 1


def test_struct_layouts_match_header():
    # zo_panel: int + 3 pointers; zo_update_item: 2 ints + 8 pointers.
    assert ctypes.sizeof(Panel) == 32
    assert ctypes.sizeof(UpdateItem) == 8 + 8 * 8


def _detail():
    return zo.lib().zo_last_error_detail().decode()


def test_status_strings():
    L = zo.lib()
    assert L.zo_status_str(0) == b"ok"
    assert L.zo_status_str(6) == b"workspace too small"


@pytest.mark.parametrize("args,needle", [
    (dict(T=0), "T, m, n"),
    (dict(r=0), "r = 0"),
    (dict(r=129), "r = 129"),
    (dict(q=0), "q = 0"),
    (dict(nblk=257), "nblk = 257"),
    (dict(m=12), "m % 8"),
    (dict(n=20), "n % 8"),
    (dict(xs=5), "x_block_stride"),
    (dict(blk_query=[0, 5]), "blk_query[1]"),
    (dict(blk_sign=[1, 2]), "blk_sign[1]"),
    (dict(in_dtype=7), "in_dtype"),
    (dict(in_dtype=3), "in_dtype"),
    (dict(in_dtype=2, m=12), "m % 8"),      # fp16 shares the 16-bit limits
    (dict(in_dtype=2, xs=1028), "x_block_stride"),
])
def test_perturbed_linear_validation(args, needle):
    p = dict(T=16, m=32, n=64, r=4, q=2, nblk=2, blk_query=[0, 1], blk_sign=[1, -1], xs=0, in_dtype=1)
    p.update(args)
    nb = p["nblk"]
    bq = (ctypes.c_int * max(nb, 2))(*(p["blk_query"] + [0] * (max(nb, 2) - 2)))
    bs = (ctypes.c_int8 * max(nb, 2))(*(p["blk_sign"] + [1] * (max(nb, 2) - 2)))
    fake = 1 << 20  # never dereferenced: validation fails first
    st = zo.lib().zo_perturbed_linear(p["T"], p["m"], p["n"], p["r"], p["q"], nb, bq, bs, 1e-3,
                                      p["in_dtype"], fake, p["xs"], fake, fake, fake, fake, 1, fake,
                                      fake, 1 << 30, None)
    assert st == 1, (st, _detail())
    assert needle in _detail()


def test_perturbed_linear_rejects_small_workspace_and_nulls():
    L = zo.lib()
    bq = (ctypes.c_int * 2)(0, 0)
    bs = (ctypes.c_int8 * 2)(1, -1)
    fake = 1 << 20
    need = L.zo_perturbed_linear_workspace(16, 32, 64, 4, 1, 2, 0, 1)
    assert need > 0
    st = L.zo_perturbed_linear(16, 32, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, fake, fake, fake, fake, 1,
                               fake, fake, need - 1, None)
    assert st == 6 and "workspace" in _detail()
    st = L.zo_perturbed_linear(16, 32, 64, 4, 1, 2, bq, bs, 1e-3, 1, None, 0, fake, fake, fake, fake, 1,
                               fake, fake, need, None)
    assert st == 1 and "NULL" in _detail()
    # fp32 inputs with bf16 output is unsupported
    st = L.zo_perturbed_linear(16, 32, 64, 4, 1, 2, bq, bs, 1e-3, 0, fake, 0, fake, fake, fake, fake, 1,
                               fake, fake, need, None)
    assert st == 2
    # The output is the input type or fp32: fp16 in with bf16 out, bf16 in with fp16 out are not.
    need16 = L.zo_perturbed_linear_workspace(16, 32, 64, 4, 1, 2, 0, 2)
    assert need16 == need  # fp16 takes the same workspace layout as bf16
    for in_dt, out_dt in ((2, 1), (1, 2)):
        st = L.zo_perturbed_linear(16, 32, 64, 4, 1, 2, bq, bs, 1e-3, in_dt, fake, 0, fake, fake, fake, fake,
                                   out_dt, fake, fake, need, None)
        assert st == 2 and "out_dtype" in _detail()


def test_shared_x_workspace_holds_the_base():
    """With one X shared by several blocks the workspace also holds the fp32 T x m product
    X W^T that every block's output starts from; a single block, or per-block X, does not."""
    L = zo.lib()
    T, m, n, r, q = 300, 264, 200, 16, 2
    for dt in (0, 1, 2):
        one = L.zo_perturbed_linear_workspace(T, m, n, r, q, 1, 0, dt)
        shared = L.zo_perturbed_linear_workspace(T, m, n, r, q, 4, 0, dt)
        per_block = L.zo_perturbed_linear_workspace(T, m, n, r, q, 4, T * n, dt)
        rp = (r + 31) // 32 * 32 if dt else (r + 15) // 16 * 16
        bp_growth = 3 * m * (3 * rp * 2 if dt else rp * 4)  # the three more blocks' right factors
        assert shared - one >= T * m * 4 + bp_growth - 1024, dt
        assert shared - one <= T * m * 4 + bp_growth + 1024, dt
        assert per_block > one


def test_lora_validation_and_workspace():
    """The LoRA entry points share the full-tuning plan at rank rl + r and reject bad ranks,
    non-finite scale and NULL adapter tensors before launching anything."""
    L = zo.lib()
    bq = (ctypes.c_int * 2)(0, 0)
    bs = (ctypes.c_int8 * 2)(1, -1)
    fake = 1 << 20
    need = L.zo_lora_perturbed_linear_workspace(16, 32, 64, 8, 4, 1, 2, 0, 1)
    assert need == L.zo_perturbed_linear_workspace(16, 32, 64, 12, 1, 2, 0, 1) > 0
    assert L.zo_lora_perturbed_linear_workspace(16, 32, 64, 120, 9, 1, 2, 0, 1) == 0
    f8 = [fake] * 8
    st = L.zo_lora_perturbed_linear(16, 32, 64, 0, 4, 1, 2, bq, bs, 1e-3, 2.0, 1, fake, 0, fake, *f8, 1,
                                    fake, fake, need, None)
    assert st == 1 and "r_L" in _detail()
    st = L.zo_lora_perturbed_linear(16, 32, 64, 8, 4, 1, 2, bq, bs, 1e-3, float("inf"), 1, fake, 0, fake,
                                    *f8, 1, fake, fake, need, None)
    assert st == 1 and "scale" in _detail()
    f8n = [fake] * 4 + [None] + [fake] * 3
    st = L.zo_lora_perturbed_linear_prepare(16, 32, 64, 8, 4, 1, 2, bq, bs, 1e-3, 2.0, 1, fake, 0, *f8n,
                                            fake, need, None)
    assert st == 1 and "NULL" in _detail()
    st = L.zo_lora_perturbed_linear_prepare(16, 32, 64, 8, 4, 1, 2, bq, bs, 1e-3, 2.0, 1, fake, 0, *f8,
                                            fake, need - 1, None)
    assert st == 6


def test_refresh_validation():
    L = zo.lib()
    fake = 1 << 20
    arr = (Panel * 2)(Panel(10, fake, fake, None), Panel(3, fake, fake, None))
    assert L.zo_subspace_refresh(2, arr, 4, None, fake, 1 << 30, None) == 1
    assert "rows = 3 < r = 4" in _detail()
    assert L.zo_subspace_refresh(1, arr, 129, None, fake, 1 << 30, None) == 1  # above the rank limit
    assert L.zo_subspace_refresh(1, arr, 0, None, fake, 1 << 30, None) == 1
    assert L.zo_subspace_refresh_workspace(1, arr, 4) > 0
    assert L.zo_subspace_refresh(1, arr, 4, None, fake, 16, None) == 6


def test_refresh_workspace_size():
    """The refresh workspace as zo.h states it: 72 bytes per panel for the call's descriptor table,
    then per panel of r <= 64 one float64 r_p x r_p partial Gram matrix per 2048-row chunk and three
    r_p x r_p float64 factors (r_p = r rounded up to 16); each piece 256-byte aligned."""
    L = zo.lib()
    fake = 1 << 20
    al = lambda b: (b + 255) // 256 * 256
    for r, rows in ((64, [5000, 64, 2048, 2049]), (4, [8, 27648]), (24, [24, 100])):
        rp = (r + 15) // 16 * 16
        arr = (Panel * len(rows))(*[Panel(rw, fake, fake, None) for rw in rows])
        want = al(72 * len(rows)) + sum(al(-(-rw // 2048) * rp * rp * 8) + 3 * al(rp * rp * 8) for rw in rows)
        assert L.zo_subspace_refresh_workspace(len(rows), arr, r) == want, (r, rows)


def test_update_validation():
    L = zo.lib()
    fake = 1 << 20
    it = UpdateItem(8, 12, fake, fake, fake, fake, fake, fake, None, None)
    arr = (UpdateItem * 1)(it)
    assert L.zo_subspace_adam_update(1, arr, 1, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "n % 8" in _detail()
    it2 = UpdateItem(8, 16, fake, fake, fake, fake, fake, fake, None, None)
    arr2 = (UpdateItem * 1)(it2)
    assert L.zo_subspace_adam_update(1, arr2, 1, 4, 2, fake, 0, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "t = 0" in _detail()
    assert L.zo_subspace_adam_update(1, arr2, 1, 4, 2, fake, 1, 1e-2, 1.0, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    wide = (UpdateItem * 1)(UpdateItem(8, (1 << 20) + 8, fake, fake, fake, fake, fake, fake, None, None))
    assert L.zo_subspace_adam_update(1, wide, 1, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "n <=" in _detail()
    need = L.zo_subspace_adam_update_workspace(1, arr2, 4, 2, 1)
    assert need > 0
    # fp16 W: the same limits and workspace as bf16; other dtypes rejected.
    assert L.zo_subspace_adam_update_workspace(1, arr2, 4, 2, 2) == need
    assert L.zo_subspace_adam_update(1, arr, 2, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "n % 8" in _detail()
    assert L.zo_subspace_adam_update(1, arr2, 3, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "w_dtype" in _detail()
    assert L.zo_subspace_adam_update(1, arr2, 1, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     need - 1, None) == 6


def test_sgd_update_validation():
    """The SGD update accepts NULL moments (the Adam update does not) and checks the rest alike."""
    L = zo.lib()
    fake = 1 << 20
    no_mom = UpdateItem(8, 16, fake, fake, fake, fake, None, None, None, None)
    arr = (UpdateItem * 1)(no_mom)
    need = L.zo_subspace_sgd_update_workspace(1, arr, 4, 2, 1)
    assert need > 0
    assert L.zo_subspace_adam_update_workspace(1, arr, 4, 2, 1) == 0
    assert L.zo_subspace_adam_update(1, arr, 1, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, fake,
                                     1 << 30, None) == 1
    assert "moment" in _detail()
    assert L.zo_subspace_sgd_update(1, arr, 1, 4, 2, fake, float("nan"), None, fake, 1 << 30, None) == 1
    assert "lr" in _detail()
    assert L.zo_subspace_sgd_update(1, arr, 1, 4, 2, fake, 1e-2, None, fake, need - 1, None) == 6


def test_loss_validation():
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_sq_loss(0, 4, 4, 0, fake, fake, fake, fake, 1 << 20, None) == 1
    assert L.zo_sq_loss(2, 4, 4, 3, fake, fake, fake, fake, 1 << 20, None) == 1
    assert "dtype" in _detail()
    assert L.zo_combine_central(2, fake, 0.0, fake, None) == 1
    assert L.zo_sq_loss_workspace(2, 64, 256) > 0


def test_decoder_entry_points_validation():
    """Layer norm, attention, the fused-epilogue apply and the decoder layer reject bad
    arguments before launching anything (no GPU touched)."""
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_layernorm(4, 12, 1, fake, fake, fake, 1e-5, fake, None) == 1 and "d % 8" in _detail()
    assert L.zo_layernorm(4, 16, 5, fake, fake, fake, 1e-5, fake, None) == 1 and "dtype" in _detail()
    assert L.zo_layernorm(4, 16, 1, fake, fake, fake, -1.0, fake, None) == 1 and "eps_ln" in _detail()
    assert L.zo_layernorm(0, 16, 1, None, None, None, 1e-5, None, None) == 0  # nothing to do
    assert L.zo_causal_attention(1, 100, 30, 256, 2, 1, fake, fake, fake, fake, None) == 1
    assert "seq_len" in _detail()
    assert L.zo_causal_attention(1, 128, 64, 256, 8, 1, fake, fake, fake, fake, None) == 2  # dh = 32
    assert "head dim" in _detail()
    assert L.zo_causal_attention(1, 128, 64, 256, 2, 0, fake, fake, fake, fake, None) == 2  # fp32
    assert L.zo_causal_attention(1, 128, 64, 256, 2, 1, None, fake, fake, fake, None) == 1
    # apply_ex: bad epilogue; residual without R; misaligned residual stride
    bq = (ctypes.c_int * 2)(0, 0)
    bs = (ctypes.c_int8 * 2)(1, -1)
    need = L.zo_perturbed_linear_workspace(16, 32, 64, 4, 1, 2, 0, 1)
    st = L.zo_perturbed_linear_apply_ex(16, 32, 64, 4, 1, 2, 1, fake, 0, fake, 1, fake, 7, None, 0, fake, need,
                                        None)
    assert st == 1 and "epilogue" in _detail()
    st = L.zo_perturbed_linear_apply_ex(16, 32, 64, 4, 1, 2, 1, fake, 0, fake, 1, fake, 2, None, 0, fake, need,
                                        None)
    assert st == 1 and "NULL R" in _detail()
    st = L.zo_perturbed_linear_apply_ex(16, 32, 64, 4, 1, 2, 1, fake, 0, fake, 1, fake, 2, fake, 514, fake, need,
                                        None)
    assert st == 1 and "r_block_stride" in _detail()
    # decoder layer: sizes, dtype, block layout of H
    assert L.zo_decoder_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 1) > 0
    assert L.zo_decoder_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 2) > 0
    assert L.zo_decoder_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 0) == 0   # fp32: no attention kernel
    assert L.zo_decoder_layer_workspace(128, 60, 256, 2, 512, 8, 2, 4, 1) == 0   # T % seq_len
    assert L.zo_decoder_layer_workspace(128, 64, 256, 2, 500, 8, 2, 4, 1) == 0   # ffn % 8
    layer = zo._lib.DecoderLayerDesc()
    bq4 = (ctypes.c_int * 4)(0, 0, 1, 1)
    bs4 = (ctypes.c_int8 * 4)(1, -1, 1, -1)
    st = L.zo_decoder_layer_forward(128, 64, 256, 2, 512, 8, 2, 4, bq4, bs4, 1e-3, 1e-5, 1, fake, 0,
                                    ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "NULL" in _detail()  # the matrices of the layer are NULL
    st = L.zo_decoder_layer_forward(128, 64, 256, 2, 512, 8, 2, 4, bq4, bs4, 1e-3, 1e-5, 1, fake, 5,
                                    ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "h_block_stride" in _detail()


def test_llama_entry_points_validation():
    """RMS norm, rotary positions and the LLaMA-family layer reject bad arguments before
    launching anything (no GPU touched)."""
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_rmsnorm(4, 12, 1, fake, fake, 1e-6, fake, None) == 1 and "d % 8" in _detail()
    assert L.zo_rmsnorm(4, 16, 7, fake, fake, 1e-6, fake, None) == 1 and "dtype" in _detail()
    assert L.zo_rmsnorm(4, 16, 1, fake, fake, float("nan"), fake, None) == 1 and "eps" in _detail()
    assert L.zo_rmsnorm(4, 16, 1, fake, None, 1e-6, fake, None) == 1 and "NULL" in _detail()
    assert L.zo_rmsnorm(4, 16, 1, fake + 2, fake, 1e-6, fake, None) == 1 and "aligned" in _detail()
    assert L.zo_rope(100, 30, 256, 2, 1, fake, 1e4, None) == 1 and "seq_len" in _detail()
    assert L.zo_rope(64, 64, 256, 32, 1, fake, 1e4, None) == 1 and "head dim" in _detail()  # dh = 8
    assert L.zo_rope(0, 64, 240, 3, 1, None, 1e4, None) == 0   # dh = 80 passes the checks (nothing to do)
    assert L.zo_rope(64, 64, 256, 2, 1, fake, 1.0, None) == 1 and "base" in _detail()
    assert L.zo_rope(64, 64, 256, 2, 0, fake, 1e4, None) == 2 and "dtype" in _detail()  # fp32
    assert L.zo_rope(64, 64, 256, 2, 1, fake + 2, 1e4, None) == 1 and "aligned" in _detail()
    assert L.zo_llama_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 1) > 0
    assert L.zo_llama_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 2) > 0
    assert L.zo_llama_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 0) == 0   # fp32: no attention kernel
    assert L.zo_llama_layer_workspace(128, 60, 256, 2, 512, 8, 2, 4, 1) == 0   # T % seq_len
    assert L.zo_llama_layer_workspace(128, 64, 256, 2, 500, 8, 2, 4, 1) == 0   # ffn % 8
    # the LLaMA workspace holds the gate output beside the decoder's buffers
    assert (L.zo_llama_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 1)
            > L.zo_decoder_layer_workspace(128, 64, 256, 2, 512, 8, 2, 4, 1))
    layer = zo._lib.LlamaLayerDesc()
    bq4 = (ctypes.c_int * 4)(0, 0, 1, 1)
    bs4 = (ctypes.c_int8 * 4)(1, -1, 1, -1)
    args = (128, 64, 256, 2, 512, 8, 2, 4, bq4, bs4, 1e-3, 1e-6, 1e4, 1, fake)
    st = L.zo_llama_layer_forward(*args, 0, ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "NULL" in _detail()  # the matrices of the layer are NULL
    st = L.zo_llama_layer_forward(*args, 5, ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "h_block_stride" in _detail()
    bad_base = args[:12] + (0.5,) + args[13:]
    st = L.zo_llama_layer_forward(*bad_base, 0, ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "base" in _detail()
    bad_rms = args[:11] + (-1.0,) + args[12:]
    st = L.zo_llama_layer_forward(*bad_rms, 0, ctypes.byref(layer), fake, fake, 1 << 40, None)
    assert st == 1 and "eps_rms" in _detail()


def test_lora_layer_and_grouped_attention_validation():
    """Grouped attention and the LoRA-scheme layer reject bad arguments before launching."""
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_causal_attention_gqa(1, 128, 64, 512, 4, 3, 1, fake, fake, fake, fake, None) == 1
    assert "kv_heads" in _detail()
    assert L.zo_causal_attention_gqa(1, 128, 64, 512, 4, 0, 1, fake, fake, fake, fake, None) == 1
    assert L.zo_causal_attention_gqa(1, 128, 64, 512, 4, -1, 1, fake, fake, fake, fake, None) == 1
    assert L.zo_llama_lora_layer_workspace(128, 64, 256, 2, 0, 512, 4, 4, 2, 4, 1) == 0
    assert L.zo_causal_attention_gqa(1, 128, 64, 512, 4, 2, 0, fake, fake, fake, fake, None) == 2  # fp32
    assert L.zo_causal_attention_gqa(1, 128, 64, 512, 4, 2, 1, fake, None, fake, fake, None) == 1
    args = (128, 64, 256, 2, 1, 512, 4, 4, 2, 4)
    assert L.zo_llama_lora_layer_workspace(*args, 1) > 0
    assert L.zo_llama_lora_layer_workspace(*args, 0) == 0                       # fp32: no attention kernel
    assert L.zo_llama_lora_layer_workspace(128, 64, 256, 2, 3, 512, 4, 4, 2, 4, 1) == 0   # heads % kv_heads
    assert L.zo_llama_lora_layer_workspace(128, 64, 256, 2, 1, 512, 100, 40, 2, 4, 1) == 0  # rl + r > 128
    layer = zo._lib.LlamaLoraLayerDesc()
    bq4 = (ctypes.c_int * 4)(0, 0, 1, 1)
    bs4 = (ctypes.c_int8 * 4)(1, -1, 1, -1)
    st = L.zo_llama_lora_layer_forward(*args, bq4, bs4, 1e-3, 2.0, 1e-6, 1e6, 1, fake, 0, ctypes.byref(layer), fake,
                                       fake, 1 << 40, None)
    assert st == 1 and "NULL" in _detail()
    st = L.zo_llama_lora_layer_forward(*args, bq4, bs4, 1e-3, 2.0, 1e-6, 1e6, 1, fake, 7, ctypes.byref(layer), fake,
                                       fake, 1 << 40, None)
    assert st == 1 and "h_block_stride" in _detail()


def test_prepare_group_validation():
    """The grouped prepare rejects bad counts, NULL descriptors and a short group workspace."""
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_perturbed_linear_group_workspace(3, 64, 256, 8, 2, 4, 64 * 256, 1) > 0
    assert L.zo_perturbed_linear_group_workspace(3, 64, 256, 8, 2, 4, 64 * 256, 0) == 0   # fp32: separate
    assert L.zo_perturbed_linear_group_workspace(1, 64, 256, 8, 2, 4, 64 * 256, 1) == 0   # one matrix
    assert L.zo_perturbed_linear_group_workspace(9, 64, 256, 8, 2, 4, 64 * 256, 1) == 0
    bq = (ctypes.c_int * 2)(0, 0)
    bs = (ctypes.c_int8 * 2)(1, -1)
    m = (ctypes.c_int * 2)(64, 64)
    ptrs = (ctypes.c_void_p * 2)(fake, fake)
    need = L.zo_perturbed_linear_workspace(16, 64, 64, 4, 1, 2, 0, 1)
    sizes = (ctypes.c_size_t * 2)(need, need)
    st = L.zo_perturbed_linear_prepare_group(0, m, 16, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, ptrs, ptrs, ptrs,
                                             ptrs, sizes, fake, 1 << 30, None)
    assert st == 1 and "count" in _detail()
    st = L.zo_perturbed_linear_prepare_group(2, m, 16, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, None, ptrs, ptrs,
                                             ptrs, sizes, fake, 1 << 30, None)
    assert st == 1 and "NULL" in _detail()
    st = L.zo_perturbed_linear_prepare_group(2, m, 16, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, ptrs, ptrs, ptrs,
                                             ptrs, sizes, fake, 16, None)
    assert st == 6 and "group workspace" in _detail()
    # Aliased workspaces (one shared buffer for both matrices) are rejected before any launch.
    gneed = L.zo_perturbed_linear_group_workspace(2, 16, 64, 4, 1, 2, 0, 1)
    ws = (ctypes.c_void_p * 2)(1 << 30, (1 << 30) + need // 2)
    gws = 1 << 34
    st = L.zo_perturbed_linear_prepare_group(2, m, 16, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, ptrs, ptrs, ptrs,
                                             ws, sizes, gws, gneed, None)
    assert st == 1 and "overlap" in _detail()
    ws = (ctypes.c_void_p * 2)(1 << 30, 1 << 31)
    st = L.zo_perturbed_linear_prepare_group(2, m, 16, 64, 4, 1, 2, bq, bs, 1e-3, 1, fake, 0, ptrs, ptrs, ptrs,
                                             ws, sizes, (1 << 31) + 256, gneed, None)
    assert st == 1 and "group workspace overlaps" in _detail()


def test_empty_calls_are_no_ops():
    """count = 0 refreshes and updates, and zero-row layer norms, succeed without launching."""
    L = zo.lib()
    fake = 1 << 20
    assert L.zo_subspace_refresh(0, None, 4, None, None, 0, None) == 0
    assert L.zo_subspace_refresh_workspace(0, None, 4) == 0
    assert L.zo_subspace_adam_update(0, None, 1, 4, 2, fake, 1, 1e-2, 0.9, 0.95, 1e-8, None, None, 0, None) == 0
    assert L.zo_subspace_sgd_update(0, None, 1, 4, 2, fake, 1e-2, None, None, 0, None) == 0
    assert L.zo_layernorm(0, 64, 1, None, None, None, 1e-5, None, None) == 0
    assert L.zo_rmsnorm(0, 64, 1, None, None, 1e-6, None, None) == 0
    assert L.zo_rope(0, 64, 256, 2, 1, None, 1e4, None) == 0


def test_refresh_noalloc_validation():
    """The no-allocation refresh validates like zo_subspace_refresh and rejects, before touching
    any device, a call whose scratch need exceeds the static scratch."""
    L = zo.lib()
    fake = 1 << 20
    arr = (Panel * 2)(Panel(10, fake, fake, None), Panel(3, fake, fake, None))
    assert L.zo_subspace_refresh_noalloc(2, arr, 4, None, None) == 1
    assert "rows = 3 < r = 4" in _detail()
    assert L.zo_subspace_refresh_noalloc(1, arr, 129, None, None) == 1
    assert L.zo_subspace_refresh_noalloc(0, None, 4, None, None) == 0
    big = (Panel * 1)(Panel(1 << 26, fake, fake, None))
    need = L.zo_subspace_refresh_workspace(1, big, 64)
    assert need > zo.ZO_NOALLOC_SCRATCH_BYTES
    assert L.zo_subspace_refresh_noalloc(1, big, 64, None, None) == 6
    assert "static scratch" in _detail() and str(need) in _detail()
