"""Shared test utilities (device transfer of bf16 bit patterns, tolerances)."""
import numpy as np
import torch

from paper_2607_20457_amd import workload


def gpu_available() -> bool:
    return torch.cuda.is_available()


def to_dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def to_dev_i32(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def f64(bits: np.ndarray) -> np.ndarray:
    return workload.bf16_bits_to_f32(bits).astype(np.float64)


# Acceptance: outputs max-abs 1e-2 and LSE max-abs 1e-3 (bf16 inputs, fp32
# accumulation), plus a relative L2 bound of 1e-2 on O because at long
# context |O| itself is of order 1e-2.
O_ATOL = 1e-2
LSE_ATOL = 1e-3
O_REL_L2 = 1e-2


def check_attention(o_gpu, lse_gpu, o_ref, lse_ref, what=""):
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    err = np.max(np.abs(o_gpu - o_ref)) if o_ref.size else 0.0
    assert err <= O_ATOL, f"{what}: O max-abs error {err}"
    nrm = np.linalg.norm(o_ref)
    if nrm > 0:
        rel = np.linalg.norm(o_gpu - o_ref) / nrm
        assert rel <= O_REL_L2, f"{what}: O relative L2 error {rel}"
    if lse_gpu is not None:
        lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
        finite = np.isfinite(lse_ref)
        assert np.array_equal(np.isfinite(lse_gpu), finite), f"{what}: LSE infinities differ"
        lerr = np.max(np.abs(lse_gpu[finite] - lse_ref[finite])) if finite.any() else 0.0
        assert lerr <= LSE_ATOL, f"{what}: LSE max-abs error {lerr}"


def check_attention_bf16(o_gpu_bf16, o_ref, what=""):
    """A bf16 output is the fp32 result rounded once: the O bounds widen by
    half a bf16 ulp of the reference value (2^-9 relative)."""
    o = np.asarray(o_gpu_bf16, dtype=np.float64)
    err = np.abs(o - o_ref)
    bound = O_ATOL + np.abs(o_ref) * 2.0 ** -9
    assert np.all(err <= bound), f"{what}: O error {np.max(err - bound) + O_ATOL} above bound"
    nrm = np.linalg.norm(o_ref)
    if nrm > 0:
        rel = np.linalg.norm(o - o_ref) / nrm
        assert rel <= O_REL_L2 + 2.0 ** -9, f"{what}: O relative L2 error {rel}"
