"""Host-side checks of the C ABI: the library loads, exports every symbol include/pcmoe.h
declares, sizes workspaces, and rejects bad arguments with the documented status before any
HIP call (no GPU is touched here)."""
import ctypes
import os
import re

import pytest

from paper_2506_02965_amd import pcmoe as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(P.LIB_PATH), reason="libpcmoe.so not built")


def declared_functions():
    src = open(os.path.join(ROOT, "include", "pcmoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(moe_\w+)\s*\(", src, flags=re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 16, names
    assert sorted(P.EXPORTS) == names
    L = P.lib()
    for n in names:
        assert hasattr(L, n), n


def desc(**kw):
    base = dict(T=256, d_model=256, d_ff=512, n_experts=8, top_k=2)
    base.update(kw)
    return P.make_desc(**base)


def test_status_strings():
    assert P.status_string(P.MOE_OK) == "MOE_OK"
    assert P.status_string(P.MOE_ERR_WORKSPACE_TOO_SMALL) == "MOE_ERR_WORKSPACE_TOO_SMALL"


def test_workspace_sizes():
    d = desc(n_shared=1)
    R = 256 * 2 + 256
    assert P.moe_workspace_size(d, P.MOE_WS_FFN_SAVED) >= R * 3 * 512 * 2
    assert P.moe_workspace_size(d, P.MOE_WS_FFN_BWD) >= R * 2 * 512 * 2
    assert P.moe_workspace_size(d, P.MOE_WS_PERMUTE) > 0
    assert P.moe_workspace_size(d, P.MOE_WS_ROUTE_BWD) >= 8 * 256 * 4
    assert P.moe_workspace_size(desc(top_k=9), P.MOE_WS_PERMUTE) == 0   # invalid descriptor


FAKE = 0x1000  # never dereferenced: every call below fails validation first


@pytest.mark.parametrize("kw,status", [
    (dict(top_k=0), P.MOE_ERR_INVALID_ARGUMENT),
    (dict(top_k=9, n_experts=16), P.MOE_ERR_UNSUPPORTED),
    (dict(top_k=3, n_experts=2), P.MOE_ERR_INVALID_ARGUMENT),
    (dict(local_begin=6, local_count=4), P.MOE_ERR_INVALID_ARGUMENT),
    (dict(d_model=192), P.MOE_ERR_UNSUPPORTED),
    (dict(d_ff=100), P.MOE_ERR_UNSUPPORTED),
    (dict(n_experts=300), P.MOE_ERR_UNSUPPORTED),
    (dict(dtype="bf16", renormalize=True, T=0), P.MOE_ERR_INVALID_ARGUMENT),
    # a shard without a hosted routed expert (shared experts only) is refused: there are no offsets to read
    (dict(local_begin=0, local_count=0, n_shared=1), P.MOE_ERR_INVALID_ARGUMENT),
    # 32-bit operand extents of the grouped GEMMs: one group's dG|dU rows (T * 2 d_ff * 2 bytes) ...
    (dict(T=65536, d_model=128, d_ff=16384, n_experts=1, top_k=1, dtype="bf16"), P.MOE_ERR_UNSUPPORTED),
    (dict(T=131072, d_model=4096, d_ff=14336, n_experts=8, top_k=2, dtype="bf16"), P.MOE_ERR_UNSUPPORTED),
    # ... one group's x rows when d_model > 2 d_ff, and one expert's weight matrix
    (dict(T=262144, d_model=4096, d_ff=128, n_experts=8, top_k=2, dtype="bf16"), P.MOE_ERR_UNSUPPORTED),
    (dict(T=64, d_model=32768, d_ff=32768, n_experts=8, top_k=2, dtype="bf16"), P.MOE_ERR_UNSUPPORTED),
])
def test_descriptor_validation(kw, status):
    d = desc(**kw)
    with pytest.raises(P.MoeError) as ei:
        P.moe_combine(d, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == status


def test_extent_limits_admit_the_workloads():
    """The 2 GiB operand-extent bound leaves every benchmark workload, and the shapes just below it, accepted."""
    from paper_2506_02965_amd.synth import CONFIGS
    for c in CONFIGS.values():
        d = P.make_desc(c.T, c.d, c.f, c.E, c.k, c.local_begin, c.n_local, c.n_shared, c.renormalize, c.dtype)
        assert P.moe_workspace_size(d, P.MOE_WS_FFN_SAVED) > 0, c.name
    # largest T for d_ff = 14336 in bf16: (T + 256) * 2 * 14336 * 2 < 2^31
    t_max = ((1 << 31) - 1) // (4 * 14336) - 256
    ok = desc(T=t_max, d_model=4096, d_ff=14336, n_experts=8, top_k=2, dtype="bf16")
    assert P.moe_workspace_size(ok, P.MOE_WS_FFN_SAVED) > 0
    over = desc(T=t_max + 1, d_model=4096, d_ff=14336, n_experts=8, top_k=2, dtype="bf16")
    assert P.moe_workspace_size(over, P.MOE_WS_FFN_SAVED) == 0


def test_permute_noalloc_refuses_beyond_its_scratch():
    """The allocation-free dispatch has a fixed 1 MiB scratch: ceil(T*k / 1024) * local_count * 4 bytes must fit."""
    ok = desc(T=262144, d_model=128, d_ff=128, n_experts=256, top_k=4)        # 1024 blocks x 256 experts: 1 MiB
    with pytest.raises(P.MoeError) as ei:
        P.moe_permute_noalloc(ok, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, stream=0)   # refused for x_perm only
    assert ei.value.status == P.MOE_ERR_INVALID_ARGUMENT and "x_perm" in P.last_error()
    big = desc(T=262144 + 256, d_model=128, d_ff=128, n_experts=256, top_k=4)  # 1025 blocks
    with pytest.raises(P.MoeError) as ei:
        P.moe_permute_noalloc(big, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == P.MOE_ERR_UNSUPPORTED and "scratch" in P.last_error()


def test_null_pointers_and_workspace():
    d = desc()
    with pytest.raises(P.MoeError) as ei:
        P.moe_route(d, None, FAKE, None, 1, FAKE, FAKE, FAKE, stream=0)
    assert ei.value.status == P.MOE_ERR_INVALID_ARGUMENT and "x" in P.last_error()
    with pytest.raises(P.MoeError) as ei:
        P.moe_route(d, FAKE, FAKE, FAKE, 3, FAKE, FAKE, FAKE, stream=0)   # 3 does not divide T=256
    assert ei.value.status == P.MOE_ERR_INVALID_ARGUMENT
    need = P.moe_workspace_size(d, P.MOE_WS_PERMUTE)
    with pytest.raises(P.MoeError) as ei:
        P.moe_permute(d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, stream=0)
    assert ei.value.status == P.MOE_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(P.MoeError) as ei:
        P.moe_expert_ffn_bwd(d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                             FAKE, 0, stream=0)
    assert ei.value.status == P.MOE_ERR_WORKSPACE_TOO_SMALL
    # the router adjoint needs every expert's gate gradient: a party shard is refused
    shard = desc(n_experts=8, local_begin=0, local_count=4)
    with pytest.raises(P.MoeError) as ei:
        P.moe_route_bwd(shard, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, stream=0)
    assert ei.value.status == P.MOE_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("kw,ptrs,status", [
    (dict(lr=0.0), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(lr=float("nan")), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(weight_decay=-1.0), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(beta1=1.0), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(beta2=-0.1), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(eps=0.0), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(step=0), {}, P.MOE_ERR_INVALID_ARGUMENT),
    (dict(), dict(m=None), P.MOE_ERR_INVALID_ARGUMENT),            # AdamW needs its moments
    (dict(), dict(master=FAKE + 8), P.MOE_ERR_INVALID_ARGUMENT),   # misaligned master
    (dict(kind="sgd", lr=-1.0), dict(m=None, v=None), P.MOE_ERR_INVALID_ARGUMENT),
])
def test_update_validation(kw, ptrs, status):
    args = dict(master=None, m=FAKE, v=FAKE)
    args.update(ptrs)
    with pytest.raises(P.MoeError) as ei:
        P.moe_expert_update(desc(), P.make_opt(**kw), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0, **args)
    assert ei.value.status == status


def test_update_rejects_bad_kind():
    o = P.make_opt()
    o.kind = 7
    with pytest.raises(P.MoeError) as ei:
        P.moe_expert_update(desc(), o, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, stream=0)
    assert ei.value.status == P.MOE_ERR_INVALID_ARGUMENT


def test_timing_report_empty():
    P.moe_kernel_timing(False)
    P.moe_kernel_timing_select("gemm_bwd_dx")
    P.moe_kernel_timing_select(None)
    assert P.moe_kernel_timing_report() == {}


def test_training_footprint_scales_expert_state_only():
    """One party's expert-layer memory: the hosted experts' state scales with the number hosted, the row-space
    buffers do not (their capacity is T*k rows either way)."""
    import dataclasses
    from paper_2506_02965_amd.layer import training_footprint
    from paper_2506_02965_amd.synth import CONFIGS
    cfg = dataclasses.replace(CONFIGS[3], bias=None, router_backward=True, local_begin=0)
    f64, f8 = training_footprint(cfg, 64), training_footprint(cfg, 8)
    assert f64["expert_state"] == 8 * f8["expert_state"]
    assert f64["expert_state"] == 64 * 3 * 1408 * 2048 * (2 + 2 + 12)
    assert abs(f64["activations"] - f8["activations"]) < 1e-3 * f64["activations"]
    assert f64["owner"] == f8["owner"]


def test_binding_refuses_host_and_strided_tensors():
    """The binding hands device addresses to the library: a host tensor, or a view whose elements are not dense,
    is refused before any call is made."""
    import torch
    d = desc()
    x = torch.zeros(256, 256)
    with pytest.raises(ValueError, match="GPU tensor"):
        P.moe_route(d, x, FAKE, None, 1, FAKE, FAKE, FAKE, stream=0)

    class StridedDeviceView:  # stands in for a non-contiguous GPU tensor without a GPU
        is_cuda = True
        shape = (256, 128)

        def is_contiguous(self):
            return False

        def stride(self):
            return (256, 2)

    with pytest.raises(ValueError, match="contiguous"):
        P.moe_route(d, StridedDeviceView(), FAKE, None, 1, FAKE, FAKE, FAKE, stream=0)


def test_header_compiles_as_c(tmp_path):
    """include/pcmoe.h is a C header: a C11 translation unit that includes it and uses its types and calls
    compiles with no diagnostic from the header itself."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("gcc or the ROCm headers are not available")
    src = tmp_path / "abi_check.c"
    src.write_text('#include "pcmoe.h"\n'
                   "int main(void) {\n"
                   "  moe_desc d = {0};\n"
                   "  moe_opt o = {0};\n"
                   "  (void)o;\n"
                   "  return moe_route(&d, 0, 0, 0, 1, 0, 0, 0, 0) == MOE_OK ? 0 : (int)moe_status_string(MOE_OK)[0];\n"
                   "}\n")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                        "-I/opt/rocm/include", "-I" + os.path.join(ROOT, "include"), str(src)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert "pcmoe.h" not in r.stderr, r.stderr
