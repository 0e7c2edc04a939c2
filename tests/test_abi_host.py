"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host-side sizing and validation behave as documented.  No call here
reaches the GPU."""
import ctypes as C
import os
import re

import pytest

from paper_2509_15965_amd import rl_decode as R
from paper_2509_15965_amd.configs import WORKLOADS, ModelShape

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rl_decode.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rl_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    lib = R.lib()
    names = declared_functions()
    assert len(names) >= 16
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(R.EXPORTS) == names


def cfg_for(name, max_seqs=8, max_ctx=64, max_prefill=64):
    return R.make_config(WORKLOADS[name].model, max_seqs, max_ctx, max_prefill)


def test_kv_bytes_follow_documented_layout():
    for name in WORKLOADS:
        m = WORKLOADS[name].model
        c = cfg_for(name, max_seqs=3, max_ctx=50)
        cap = 64                                   # 50 rounded up to a multiple of 32
        es = 4 if m.dtype == "fp32" else 2
        assert R.kv_bytes(c) == 2 * m.n_layers * 3 * m.n_kv_heads * cap * m.head_dim * es


def test_paged_kv_bytes_follow_documented_layout():
    for name in WORKLOADS:
        m = WORKLOADS[name].model
        es = 4 if m.dtype == "fp32" else 2
        # a (layer, page, kv-head) block: 32 rows rounded up to an odd number of 256 bytes
        n = -(-32 * m.head_dim * es // 256)
        block = (n + 1 - n % 2) * 256
        # 3 slots of 50 positions in pages of 32: 2 pages each by default, or a pool of 4 pages
        c = R.make_config(m, 3, 50, 64, kv_page_size=32)
        assert R.kv_bytes(c) == 2 * m.n_layers * 6 * m.n_kv_heads * block
        c = R.make_config(m, 3, 50, 64, kv_page_size=32, kv_pages=4)
        assert R.kv_bytes(c) == 2 * m.n_layers * 4 * m.n_kv_heads * block
        # the page table travels with every call's metadata: the workspace grows with it
        assert R.workspace_bytes(c) >= R.workspace_bytes(cfg_for(name, 3, 50, 64))


def test_workspace_grows_with_capacity():
    a = R.workspace_bytes(cfg_for("qwen7b", 8, 64, 64))
    b = R.workspace_bytes(cfg_for("qwen7b", 512, 5120, 32768))
    assert 0 < a < b
    assert b % 256 == 0


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, R.RL_ERR_UNSUPPORTED),
    ("n_kv_heads", 3, R.RL_ERR_UNSUPPORTED),
    ("vocab", 1001, R.RL_ERR_UNSUPPORTED),
    ("dtype", 7, R.RL_ERR_INVALID_ARG),
    ("max_ctx", 1, R.RL_ERR_INVALID_ARG),
    ("rms_eps", 0.0, R.RL_ERR_INVALID_ARG),
    ("rope_theta", 1.0, R.RL_ERR_INVALID_ARG),
    ("reserved", 1, R.RL_ERR_INVALID_ARG),
    ("max_seqs", 0, R.RL_ERR_INVALID_ARG),
    ("kv_page_size", 48, R.RL_ERR_INVALID_ARG),      # not a multiple of 32
    ("kv_page_size", 16, R.RL_ERR_INVALID_ARG),      # below 32
    ("kv_pages", 5, R.RL_ERR_INVALID_ARG),           # pages without a page size
    ("kv_pages", -1, R.RL_ERR_INVALID_ARG),
])
def test_invalid_configs_rejected_before_any_device_call(field, value, status):
    c = cfg_for("tiny")
    setattr(c, field, value)
    assert R.kv_bytes(c) == 0
    assert R.workspace_bytes(c) == 0
    w = R.Weights(*([256] * 12))
    h = C.c_void_p(123)
    st = R.lib().rl_decode_create(C.byref(c), C.byref(w), 256, 1 << 40, 256, 1 << 40, None, C.byref(h))
    assert st == status
    assert not h.value


@pytest.mark.parametrize("fields,status", [
    ({"n_experts": 1025, "top_k": 8, "expert_ffn": 768}, R.RL_ERR_INVALID_ARG),     # too many experts
    ({"n_experts": 8, "top_k": 9, "expert_ffn": 768}, R.RL_ERR_INVALID_ARG),        # top_k > n_experts
    ({"n_experts": 64, "top_k": 17, "expert_ffn": 768}, R.RL_ERR_INVALID_ARG),      # top_k > 16
    ({"n_experts": 8, "top_k": 2, "expert_ffn": 40}, R.RL_ERR_INVALID_ARG),         # width not a multiple of 16
    ({"n_experts": 0, "top_k": 2, "expert_ffn": 0}, R.RL_ERR_INVALID_ARG),          # top_k without experts
    ({"n_experts": 8, "top_k": 2, "expert_ffn": 64, "dtype": 0}, R.RL_ERR_UNSUPPORTED),   # fp32
    ({"n_experts": 8, "top_k": 2, "expert_ffn": 64, "hidden": 8192}, R.RL_ERR_UNSUPPORTED),
])
def test_invalid_moe_configs_rejected(fields, status):
    c = cfg_for("qwen7b")
    for k, v in fields.items():
        setattr(c, k, v)
    assert R.kv_bytes(c) == 0
    w = R.Weights(*([256] * 12))
    h = C.c_void_p(123)
    st = R.lib().rl_decode_create(C.byref(c), C.byref(w), 256, 1 << 40, 256, 1 << 40, None, C.byref(h))
    assert st == status and not h.value


def test_moe_workspace_holds_the_expert_buffers():
    """The Qwen3-30B-A3B shape: the workspace adds the router logits, pair
    lists and the k planes of expert outputs ([k][rows][hidden] fp32)."""
    from paper_2509_15965_amd.configs import QWEN3_MOE
    c = R.make_config(QWEN3_MOE, 512, 2048, 4096)
    dense = R.make_config(ModelShape(**{**QWEN3_MOE.as_dict(), "n_experts": 0, "top_k": 0, "expert_ffn": 0}),
                          512, 2048, 4096)
    extra = R.workspace_bytes(c) - R.workspace_bytes(dense)
    rows, k, H, E, Fe = 4096, 8, 2048, 128, 768
    assert extra >= rows * (E * 4 + k * 12 + k * Fe * 2 + k * H * 4)
    # the MLP weights of a mixture of experts: NULL dense matrices are accepted
    w = R.Weights(*([256] * 5 + [0, 0] + [256] * 5))
    h = C.c_void_p(123)
    st = R.lib().rl_decode_create(C.byref(c), C.byref(w), 256, 1, 256, 1, None, C.byref(h))
    assert st == R.RL_ERR_CAPACITY and not h.value          # weights pass; the tiny buffers do not
    w = R.Weights(*([256] * 9 + [0, 256, 256]))              # no router
    st = R.lib().rl_decode_create(C.byref(c), C.byref(w), 256, 1 << 40, 256, 1 << 40, None, C.byref(h))
    assert st == R.RL_ERR_INVALID_ARG and not h.value


def test_bf16_weight_matrix_of_4_gib_rejected():
    """The bf16 GEMMs address a weight matrix with 32-bit byte offsets: an LM
    head of 600000 x 3584 bf16 (4.3 GB) is refused at create, 590000 is not."""
    c = cfg_for("qwen7b")
    c.vocab = 600000
    assert R.kv_bytes(c) == 0
    h = C.c_void_p(123)
    w = R.Weights(*([256] * 12))
    st = R.lib().rl_decode_create(C.byref(c), C.byref(w), 256, 1 << 40, 256, 1 << 40, None, C.byref(h))
    assert st == R.RL_ERR_UNSUPPORTED
    assert not h.value
    c.vocab = 590000
    assert R.kv_bytes(c) > 0


def test_create_validates_pointers_and_sizes_first():
    lib = R.lib()
    c = cfg_for("tiny")
    h = C.c_void_p(1)
    w = R.Weights(*([256] * 12))
    assert lib.rl_decode_create(C.byref(c), None, 256, 1 << 40, 256, 1 << 40, None, C.byref(h)) == R.RL_ERR_INVALID_ARG
    w_bad = R.Weights(*([256] * 8 + [0]))
    assert lib.rl_decode_create(C.byref(c), C.byref(w_bad), 256, 1 << 40, 256, 1 << 40, None, C.byref(h)) == R.RL_ERR_INVALID_ARG
    w_mis = R.Weights(*([256] * 8 + [258]))
    assert lib.rl_decode_create(C.byref(c), C.byref(w_mis), 256, 1 << 40, 256, 1 << 40, None, C.byref(h)) == R.RL_ERR_INVALID_ARG
    assert lib.rl_decode_create(C.byref(c), C.byref(w), 128, 1 << 40, 256, 1 << 40, None, C.byref(h)) == R.RL_ERR_INVALID_ARG
    small = R.kv_bytes(c) - 1
    assert lib.rl_decode_create(C.byref(c), C.byref(w), 256, small, 256, 1 << 40, None, C.byref(h)) == R.RL_ERR_CAPACITY
    assert lib.rl_decode_create(C.byref(c), C.byref(w), 256, 1 << 40, 256, 1 << 40, None, None) == R.RL_ERR_INVALID_ARG
    assert not h.value


def test_null_and_foreign_contexts():
    lib = R.lib()
    assert lib.rl_decode_destroy(None) == R.RL_OK
    assert lib.rl_slot_length(None, 0) == -1
    sp = R.SampleParams(1, 1.0, 0)
    assert lib.rl_decode_step(None, 1, None, None, None, None, C.byref(sp), None, None, None) == R.RL_ERR_STATE
    assert lib.rl_prefill(None, 1, 1, None, None, None, None, None, 0, None, C.byref(sp), None, None, None) == R.RL_ERR_STATE
    junk = (C.c_uint32 * 64)()
    assert lib.rl_decode_step(C.addressof(junk), 1, None, None, None, None, C.byref(sp), None, None, None) == R.RL_ERR_STATE
    assert lib.rl_release_slots(None, 0, None) == R.RL_ERR_STATE
    assert lib.rl_decode_set_option(None, 1, 0) == R.RL_ERR_STATE
    assert lib.rl_decode_last_error(None) == b"invalid or destroyed context"


def test_status_strings():
    lib = R.lib()
    for s in range(6):
        assert lib.rl_status_string(s)
    assert lib.rl_status_string(99) == b"unknown status"


def test_probe_copy_argument_checks():
    lib = R.lib()
    assert lib.rl_probe_copy(None, None, 16, None) == R.RL_ERR_INVALID_ARG
    assert lib.rl_probe_copy(256, 512, 15, None) == R.RL_ERR_INVALID_ARG
    assert lib.rl_probe_copy(258, 512, 16, None) == R.RL_ERR_INVALID_ARG


def _compile_and_run(tmp_path, body):
    """Build a C program that includes the header and prints `body`'s lines."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "abi.c"
    src.write_text('#include <stddef.h>\n#include <stdio.h>\n#include "rl_decode.h"\n'
                   "int main(void) {\n" + body + "return 0;\n}\n")
    exe = tmp_path / "abi"
    subprocess.run([cc, "-std=c11", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return dict(line.split("=") for line in out.split())


_STRUCTS = {"rl_model_config": R.ModelConfig, "rl_weights": R.Weights, "rl_sample_params": R.SampleParams,
            "rl_kernel_stats": R.KernelStats, "rl_attn_plan_stats": R.AttnPlanStats}


def test_binding_structs_match_the_header_layout(tmp_path):
    """Every ctypes mirror has the C struct's size and each field's offset, as
    the C compiler lays them out from the header."""
    body = ""
    for cname, py in _STRUCTS.items():
        body += f'printf("{cname}=%zu\\n", sizeof({cname}));\n'
        for f, _ in py._fields_:
            body += f'printf("{cname}.{f}=%zu\\n", offsetof({cname}, {f}));\n'
    got = _compile_and_run(tmp_path, body)
    for cname, py in _STRUCTS.items():
        assert int(got[cname]) == C.sizeof(py), cname
        for f, _ in py._fields_:
            assert int(got[f"{cname}.{f}"]) == getattr(py, f).offset, (cname, f)


def test_binding_constants_match_the_header_enums(tmp_path):
    """Status codes, dtypes, options, GEMM kernel codes and kernel-class
    indices of the binding equal the header's enum values."""
    names = [n for n in dir(R) if re.fullmatch(r"RL_(OK|ERR_[A-Z_]+|DTYPE_[A-Z0-9]+|OPT_[A-Z_]+|GEMM_[A-Z0-9_]+)", n)]
    assert len(names) >= 20
    body = "".join(f'printf("{n}=%d\\n", (int){n});\n' for n in names)
    classes = ["RL_K_" + k.upper() for k in R.KERNEL_CLASSES]
    body += "".join(f'printf("{k}=%d\\n", (int){k});\n' for k in classes)
    body += 'printf("RL_K_COUNT=%d\\n", (int)RL_K_COUNT);\n'
    got = _compile_and_run(tmp_path, body)
    for n in names:
        assert int(got[n]) == getattr(R, n), n
    for i, k in enumerate(classes):
        assert int(got[k]) == i, k
    assert int(got["RL_K_COUNT"]) == len(R.KERNEL_CLASSES)
