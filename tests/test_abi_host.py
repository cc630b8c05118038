"""The C ABI on the host: the library loads, exports every declared symbol,
its structs match the header's layout, and argument checks that run before
any device work return the documented codes.  No GPU needed."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pipo.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2605_27255_amd import pipo, build
    if not os.path.exists(pipo.LIB_PATH):
        build.build()
    return pipo.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(pipo_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    from paper_2605_27255_amd import pipo
    names = declared_functions()
    assert set(names) == set(pipo.EXPORTED), names
    out = subprocess.run(["nm", "-D", "--defined-only", pipo.LIB_PATH], capture_output=True, text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}$", out, re.M), f"{n} not exported"
        getattr(lib, n)


def test_struct_layout_matches_header(tmp_path):
    from paper_2605_27255_amd import pipo
    src = tmp_path / "layout.c"
    src.write_text(f'''#include <stdio.h>
#include <stddef.h>
#include "{HEADER}"
int main(void) {{
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu\\n", sizeof(pipo_config), sizeof(pipo_sampling), sizeof(pipo_pair),
         offsetof(pipo_config, gain_mode), offsetof(pipo_sampling, seeds), offsetof(pipo_pair, accept),
         offsetof(pipo_config, heads), offsetof(pipo_sampling, top_k), offsetof(pipo_sampling, rep_penalty));
  return 0;
}}''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", str(src), "-o", str(exe)], check=True)
    got = list(map(int, subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()))
    assert got == [ctypes.sizeof(pipo.PipoConfig), ctypes.sizeof(pipo.PipoSampling), ctypes.sizeof(pipo.PipoPair),
                   pipo.PipoConfig.gain_mode.offset, pipo.PipoSampling.seeds.offset, pipo.PipoPair.accept.offset,
                   pipo.PipoConfig.heads.offset, pipo.PipoSampling.top_k.offset,
                   pipo.PipoSampling.rep_penalty.offset]
    assert got[2] == 16


def _cfg(**kw):
    from paper_2605_27255_amd import pipo
    from synth.configs import TINY
    c = pipo.make_config(TINY, 1, 64, 16)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("hidden", 250), ("ffn", 1000), ("vocab", 4090),
                                         ("max_batch", 65), ("max_batch", 0), ("n_kv_heads", 3),
                                         ("prefill_chunk", 0), ("max_latent", 0), ("gain_mode", 2), ("heads", 8),
                                         ("pad_id", 5000)])
def test_bad_config_is_rejected_before_device_work(lib, field, value):
    from paper_2605_27255_amd import pipo
    ctx = ctypes.c_void_p()
    rc = lib.pipo_init_weights(ctypes.byref(_cfg(**{field: value})), 0, None, ctypes.byref(ctx))
    assert rc == pipo.PIPO_EINVAL
    assert not ctx.value
    assert lib.pipo_last_error(None)


def test_null_arguments(lib):
    from paper_2605_27255_amd import pipo
    ctx = ctypes.c_void_p()
    assert lib.pipo_init_weights(None, 0, None, ctypes.byref(ctx)) == pipo.PIPO_EINVAL
    assert lib.pipo_init_weights(ctypes.byref(_cfg()), 0, None, None) == pipo.PIPO_EINVAL
    smp = pipo.PipoSampling(0.5, 0.0, 1.0, None)
    assert lib.pipo_prefill(None, 1, None, 4, ctypes.byref(smp), None, None, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_decode_step(None, None, None, None, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_regular_prefill(None, 1, None, 4, ctypes.byref(smp), None, None, None) == pipo.PIPO_EINVAL
    # OPD targets: argument checks come before any device work
    fake = ctypes.c_void_p(16)
    assert lib.pipo_opd_teacher_rows(None, 4, 0, fake, None) == pipo.PIPO_EINVAL
    assert lib.pipo_opd_teacher_rows(fake, -1, 0, fake, None) == pipo.PIPO_EINVAL
    assert lib.pipo_opd_targets(4, 8, None, fake, 4, None, fake, fake, fake, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_opd_targets(4, 6, fake, fake, 4, None, fake, fake, fake, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_opd_targets(4, 8, ctypes.c_void_p(20), fake, 4, None, fake, fake, fake, None,
                                None) == pipo.PIPO_EINVAL
    assert lib.pipo_opd_targets(4, 8, fake, fake, 0, None, fake, fake, fake, None, None) == pipo.PIPO_EINVAL
    lens = (ctypes.c_int32 * 1)(4)
    assert lib.pipo_prefill_ragged(None, 1, None, 4, lens, ctypes.byref(smp), None, None, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_prefill_ragged(None, 1, None, 4, None, ctypes.byref(smp), None, None, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_regular_prefill_ragged(None, 1, None, 4, lens, ctypes.byref(smp), None, None,
                                           None) == pipo.PIPO_EINVAL
    assert lib.pipo_regular_step(None, None, None, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_read_weight(None, b"embed", 0, 1, None) == pipo.PIPO_EINVAL
    assert lib.pipo_free(None) == pipo.PIPO_OK
    assert b"ctx" in lib.pipo_last_error(None)
    # measurement aids: argument checks before any HIP call
    us = ctypes.c_double()
    lib.pipo_calibrate_stream.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                          ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    lib.pipo_calibrate_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    assert lib.pipo_calibrate_stream(None, 1024, 1024, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_stream(fake, 4096, 1000, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_stream(fake, 1024, 2048, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_stream(fake, 1024, 1024, 0, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_stream(fake, 1024, 1024, 1, None, None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_mfma(None, 1, 1, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_mfma(fake, 3, 1, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL
    assert lib.pipo_calibrate_mfma(fake, 1, 0, 1, ctypes.byref(us), None) == pipo.PIPO_EINVAL


def test_gemv_dispatch_refuses_unlisted_variant(lib):
    """The decode GEMV launcher has one kernel per (prologue, epilogue) pair the
    step uses; any other pair launches nothing and reports -1, which the
    runtime turns into PIPO_EINVAL for the call.  The launcher is a C++ symbol
    of the library, called here on a zeroed parameter block (an unlisted pair
    returns before reading it, with no HIP call)."""
    fn = getattr(lib, "_ZN4pipo11launch_gemvERKNS_10GemvParamsEiiP12ihipStream_t")
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    block = ctypes.create_string_buffer(4096)
    pro_f32, pro_mtp, epi_qkv, epi_logits, epi_swiglu = 1, 3, 3, 4, 2
    for pro, epi in ((pro_f32, epi_qkv), (pro_mtp, epi_logits), (pro_f32, epi_swiglu), (7, 0), (0, 9)):
        assert fn(ctypes.addressof(block), pro, epi, None) == -1, (pro, epi)
