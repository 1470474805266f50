"""The C-ABI library loads and exports every symbol include/pulse.h declares, and
host-side argument validation returns the documented status codes.  No compute
call is made here: every call below returns before touching the GPU."""
import os
import re
import subprocess

import pytest

from paper_2609_34555_amd import pulse as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pulse.h")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"PULSE_API\s+[\w\s\*]+?\b(pulse_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    decl = declared_symbols()
    assert len(decl) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = sorted(set(m.group(1) for m in re.finditer(r"\sT\s(pulse_\w+)", out)))
    assert exported == decl
    L = P.lib()
    for name in decl:
        assert hasattr(L, name)
    assert set(P.EXPORTED) == set(decl)


def test_header_compiles_as_strict_c_and_cxx():
    """include/pulse.h is a plain C header: it compiles as C99, C11 and C++17 with every warning
    an error, and a C translation unit can take the address of every declared entry point."""
    for lang, std in (("c", "c99"), ("c", "c11"), ("c++", "c++17")):
        cc = "gcc" if lang == "c" else "g++"
        subprocess.run([cc, f"-std={std}", "-Wall", "-Wextra", "-Werror", "-pedantic", "-fsyntax-only", "-x", lang,
                        HEADER], check=True)
    names = declared_symbols()
    src = '#include "pulse.h"\n' + "".join(f"void* p{i} = (void*)&{n};\n" for i, n in enumerate(names))
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only", "-I", os.path.dirname(HEADER), "-x", "c",
                    "-"], input=src, text=True, check=True)


def test_library_needs_only_the_hip_runtime():
    """libpulse.so links no BLAS or other ROCm library: every kernel, the normal batch's FFN
    GEMMs included, is built into it, so it loads wherever the HIP runtime does."""
    out = subprocess.run(["readelf", "-d", P.LIB_PATH], capture_output=True, text=True, check=True).stdout
    needed = re.findall(r"\(NEEDED\)\s+Shared library: \[([^\]]+)\]", out)
    rocm = [n for n in needed if not re.match(r"lib(c|m|dl|gcc_s|stdc\+\+|pthread|rt)\.so", n)]
    assert rocm and all(n.startswith("libamdhip64.so") for n in rocm), needed


def test_status_strings():
    for code, name in [(0, "PULSE_OK"), (4, "PULSE_ERR_POOL_EXHAUSTED"), (7, "PULSE_ERR_BAD_INDEX")]:
        assert P.status_string(code) == name


def shape(**kw):
    base = dict(num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=16, dtype=P.PULSE_BF16)
    base.update(kw)
    return P.make_shape(**base)


def test_block_and_workspace_sizes():
    assert P.pulse_block_bytes(shape()) == 64 * 1024
    assert P.pulse_block_bytes(shape(block_size=32)) == 128 * 1024
    assert P.pulse_block_bytes(shape(head_dim=64)) == 0
    assert P.pulse_block_bytes(shape(num_q_heads=30)) == 0  # not a multiple
    assert P.pulse_block_bytes(shape(num_q_heads=8 * 17)) == 0  # G > 16
    a = P.pulse_workspace_bytes(shape(), 8, 128, 16384)
    b = P.pulse_workspace_bytes(shape(), 4, 64, 8000)
    assert a > 0 and b > 0 and b <= a
    assert P.pulse_workspace_bytes(shape(), -1, 128, 10) == 0


def test_attention_workgroups():
    """Split-K workgroups per (request, KV head): one (no merge kernel) where 8 waves cover a
    selection at the ~2048-wave sizing, several otherwise; 0 for invalid arguments."""
    assert P.pulse_attention_workgroups(shape(), 32, 256) == 1  # 32 x 8 units, 8 splits of 32 blocks
    assert P.pulse_attention_workgroups(shape(), 8, 128) == 4  # 64 units, 32 splits of 4 blocks
    assert P.pulse_attention_workgroups(shape(num_q_heads=64, block_size=32), 4, 256) == 8
    assert P.pulse_attention_workgroups(shape(dtype=P.PULSE_F16), 1, 25) == 1  # 7 splits, one workgroup
    assert P.pulse_attention_workgroups(shape(num_q_heads=8 * 12), 8, 128) == 8  # G 12: 4-wave workgroups
    assert P.pulse_attention_workgroups(shape(), 0, 128) == 0
    assert P.pulse_attention_workgroups(shape(), 8, 0) == 0
    assert P.pulse_attention_workgroups(shape(head_dim=64), 8, 128) == 0


FAKE = 0x1000  # never dereferenced: every call below fails validation first


def test_select_validation_codes():
    s = shape()
    args = dict(q=FAKE, digests=FAKE, blk_off=FAKE, B=2, total_blocks=10, solo_kv_head=0, k_mid=FAKE,
                n_sink_blocks=1, n_local_blocks=8, k_max=16, sel_idx=FAKE, sel_cnt=FAKE, scores=None,
                dev_status=FAKE, ws=FAKE, ws_bytes=1, stream=0, check=False)
    assert P.pulse_select_solohead(s, **args) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_select_solohead(shape(head_dim=64), **args) == P.PULSE_ERR_UNSUPPORTED
    assert P.pulse_select_solohead(s, **{**args, "solo_kv_head": 8}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_select_solohead(s, **{**args, "k_max": 0}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_select_solohead(s, **{**args, "q": None}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_select_solohead(s, **{**args, "dev_status": None}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_select_solohead(s, **{**args, "B": 0}) == P.PULSE_OK  # nothing to do


def test_recall_and_attention_validation_codes():
    s = shape()
    r = dict(host_kv=FAKE, blk_off=FAKE, B=2, sel_idx=FAKE, sel_cnt=FAKE, k_max=16, block_table=FAKE,
             max_blocks=100, free_slots=FAKE, free_head=FAKE, n_free=10, slot_pool=FAKE, n_slots=50, stats=FAKE,
             dev_status=FAKE, ws=FAKE, ws_bytes=1, stream=0, check=False)
    assert P.pulse_recall_gather(s, **r) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_recall_gather(s, **{**r, "host_kv": None}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_recall_gather(s, **{**r, "B": 5000}) == P.PULSE_ERR_UNSUPPORTED
    assert P.pulse_recall_gather(s, **{**r, "n_slots": 0}) == P.PULSE_ERR_INVALID_ARG
    a = dict(q=FAKE, slot_pool=FAKE, n_slots=50, block_table=FAKE, max_blocks=100, sel_idx=FAKE, sel_cnt=FAKE,
             k_max=16, ctx_len=FAKE, B=2, sm_scale=0.1, out=FAKE, lse=None, dev_status=FAKE, ws=FAKE, ws_bytes=1,
             stream=0, check=False)
    assert P.pulse_sparse_decode_attn(s, **a) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_sparse_decode_attn(s, **{**a, "out": None}) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_sparse_decode_attn(shape(block_size=8), **a) == P.PULSE_ERR_UNSUPPORTED


def test_decode_layer_validation_codes():
    la = P.pulse_layer_args()
    la.shape = shape()
    la.B = 2
    la.total_blocks = 10
    for f in ("ctx_len", "blk_off", "q", "digests", "k_mid", "sel_idx", "sel_cnt", "host_kv", "block_table",
              "free_slots", "free_head", "slot_pool", "stats", "out", "dev_status", "ws"):
        setattr(la, f, FAKE)
    la.k_max, la.max_blocks, la.n_free, la.n_slots, la.n_sink_blocks, la.n_local_blocks = 16, 100, 10, 50, 1, 8
    la.ws_bytes = 1
    assert P.pulse_decode_layer(la, stream=0, check=False) == P.PULSE_ERR_WORKSPACE
    la.ws_bytes = P.pulse_workspace_bytes(la.shape, 2, 16, 10)
    la.out = None
    assert P.pulse_decode_layer(la, stream=0, check=False) == P.PULSE_ERR_INVALID_ARG
    assert P.lib().pulse_decode_layer(None, None) == P.PULSE_ERR_INVALID_ARG


def test_decode_layer_noalloc_validation_codes():
    """The static-workspace variant: a caller workspace is refused, a call needing more than
    the static array is refused before any device work, B = 0 does nothing."""
    la = P.pulse_layer_args()
    la.shape = shape()
    la.B = 2
    la.total_blocks = 10
    for f in ("ctx_len", "blk_off", "q", "digests", "k_mid", "sel_idx", "sel_cnt", "host_kv", "block_table",
              "free_slots", "free_head", "slot_pool", "stats", "out", "dev_status"):
        setattr(la, f, FAKE)
    la.k_max, la.max_blocks, la.n_free, la.n_slots, la.n_sink_blocks, la.n_local_blocks = 16, 100, 10, 50, 1, 8
    la.ws, la.ws_bytes = FAKE, 1 << 20
    assert P.pulse_decode_layer_noalloc(la, stream=0, check=False) == P.PULSE_ERR_INVALID_ARG
    la.ws, la.ws_bytes = None, 0
    # the largest total_blocks whose workspace fits, and one more block than that
    fit = (P.NOALLOC_SCRATCH_BYTES - P.pulse_workspace_bytes(la.shape, 2, 16, 0)) // 4
    assert P.pulse_workspace_bytes(la.shape, 2, 16, fit) <= P.NOALLOC_SCRATCH_BYTES
    la.total_blocks = fit + 256
    assert P.pulse_workspace_bytes(la.shape, 2, 16, la.total_blocks) > P.NOALLOC_SCRATCH_BYTES
    assert P.pulse_decode_layer_noalloc(la, stream=0, check=False) == P.PULSE_ERR_WORKSPACE
    la.total_blocks = 10
    la.shape = shape(head_dim=64)
    assert P.pulse_decode_layer_noalloc(la, stream=0, check=False) == P.PULSE_ERR_UNSUPPORTED
    la.shape = shape()
    la.B = 0
    assert P.pulse_decode_layer_noalloc(la, stream=0, check=False) == P.PULSE_OK
    assert P.lib().pulse_decode_layer_noalloc(None, None) == P.PULSE_ERR_INVALID_ARG
    text = open(HEADER).read()
    assert re.search(r"#define PULSE_NOALLOC_SCRATCH_BYTES \(\(size_t\)32 << 20\)", text)
    assert P.NOALLOC_SCRATCH_BYTES == 32 << 20


def test_probe_and_baseline_validation():
    assert P.pulse_probe_host_read(FAKE, FAKE, 1000, stream=0, check=False) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_baseline_memcpy_units(FAKE, FAKE, FAKE, FAKE, 0, 4096, stream=0, check=False) == P.PULSE_OK
    assert P.pulse_baseline_memcpy_units(None, FAKE, FAKE, FAKE, 3, 4096, stream=0, check=False) == \
        P.PULSE_ERR_INVALID_ARG


def test_new_entry_points_validation_codes():
    sh = shape()
    # B above the supported maximum
    assert P.pulse_release_recalled(sh, 4097, 16, 10, FAKE, 100, FAKE, FAKE, FAKE, FAKE, 1 << 30, stream=0,
                                    check=False) == P.PULSE_ERR_UNSUPPORTED
    assert P.pulse_release_recalled(sh, 2, 16, 10, FAKE, 100, FAKE, FAKE, FAKE, FAKE, 1, stream=0,
                                    check=False) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_release_recalled(sh, 0, 16, 10, None, 100, None, None, None, None, 0, stream=0,
                                    check=False) == P.PULSE_OK
    assert P.pulse_select_average(sh, FAKE, FAKE, FAKE, 2, 10, FAKE, 1, 8, 16, FAKE, FAKE, None, FAKE, FAKE, 1,
                                  stream=0, check=False) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_mam(sh, FAKE, FAKE, 10, FAKE, 0, FAKE, 2, 1, 8, 0.1, FAKE, FAKE, FAKE, 1 << 30, stream=0,
                       check=False) == P.PULSE_ERR_INVALID_ARG
    assert P.pulse_mam(sh, FAKE, FAKE, 10, FAKE, 100, FAKE, 2, 1, 8, 0.1, FAKE, FAKE, FAKE, 1, stream=0,
                       check=False) == P.PULSE_ERR_WORKSPACE
    assert P.pulse_probe_hbm_read(FAKE, 1000, FAKE, stream=0, check=False) == P.PULSE_ERR_INVALID_ARG
    assert P.lib().pulse_irq_step(None, None, 1, None, 0, 0, 1, None, None, None) == P.PULSE_ERR_INVALID_ARG
    la = P.pulse_layer_args()
    la.shape = sh
    la.B = 4097
    la.k_max, la.max_blocks, la.n_free, la.n_slots, la.n_sink_blocks, la.n_local_blocks = 16, 100, 10, 50, 1, 8
    assert P.pulse_decode_layer(la, stream=0, check=False) == P.PULSE_ERR_UNSUPPORTED


def test_oracle_and_product_share_nothing():
    """The oracle never imports the GPU package and the GPU package never imports the oracle."""
    pkg = os.path.join(ROOT, "paper_2609_34555_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in re.findall(r"(?:import|from)\s+(\w+)", txt), f
                assert "pulse_oracle" not in txt, f
    for f in os.listdir(os.path.join(ROOT, "oracle")):
        if f.endswith((".py", ".c", ".h")):
            txt = open(os.path.join(ROOT, "oracle", f)).read()
            assert "paper_2609_34555_amd" not in re.findall(r"(?:import|from)\s+([\w.]+)", txt), f
            assert "#include" not in txt or ("pulse_internal" not in txt and "pulse.h\"" not in txt), f


def test_binding_structs_match_the_header_layout(tmp_path):
    """Every struct the binding passes by pointer has the header's size and field offsets
    (compiled from include/pulse.h with the host C compiler)."""
    import ctypes
    import shutil
    import subprocess

    from paper_2609_34555_amd import pulse as P

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    structs = [P.pulse_shape, P.pulse_recall_stats, P.pulse_ioaa_params, P.pulse_layer_args,
               P.pulse_normal_layer, P.pulse_irq_stats]
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "pulse.h"', "int main(void) {"]
    for cls in structs:
        name = cls.__name__
        lines.append(f'printf("{name} size %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run([cc, "-std=c99", "-I", inc, str(src), "-o", str(exe)], check=True, capture_output=True)
    got = {}
    for line in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        name, field, value = line.split()
        got[(name, field)] = int(value)
    for cls in structs:
        name = cls.__name__
        assert got[(name, "size")] == ctypes.sizeof(cls), name
        for f, _ in cls._fields_:
            assert got[(name, f)] == getattr(cls, f).offset, (name, f)
