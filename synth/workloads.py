"""Workload shapes of the coded matrix-multiplication benchmarks.

Shapes follow the paper's experiments in spirit (Sec. III-F draws random dense
matrices and multiplies them by a vector) at sizes that fill one MI355X.
"""
from __future__ import annotations

from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    n: int
    k: int
    q: int
    r: int
    s: int
    dtype: str            # "f32" or "bf16": dtype of A, X and the parity coefficients
    seed: int
    units: int            # products / calls / decodes / iterations in one run
    a_std: float = 1.0
    extra: dict = field(default_factory=dict)

    @property
    def qb(self) -> int:
        return -(-self.q // self.k)


WORKLOADS = {
    "mds4x2_2048x512": Workload("mds4x2_2048x512", 4, 2, 2048, 512, 1, "f32", 0, 100,
                                extra={"seeds": list(range(100))}),
    "gemv16x12_65536x8192": Workload("gemv16x12_65536x8192", 16, 12, 65536, 8192, 1, "f32", 2, 1000),
    # The GEMV regime with a certified generator: of 3000 seeded N(0,1) parity
    # matrices (synth.conditioned_parity_matrix(16, 12, 2, 3000)), candidate
    # 2841 has the smallest worst decode condition number, 679 over every
    # survivor set (the plain seed-2 draw: 4589), which lets the parity be
    # stored in one fp32 plane.
    "gemv16x12_conditioned_65536x8192": Workload("gemv16x12_conditioned_65536x8192", 16, 12, 65536, 8192, 1,
                                                 "f32", 2, 1000,
                                                 extra={"parity_candidate": 2841, "candidates": 3000,
                                                        "worst_condition": 679.2, "planes": 1}),
    # The GEMV workload with 6-byte parity elements: the fp32 hi plane and a
    # bfloat16 lo plane (planes code 3), same generator and inputs.
    "gemv16x12_bf16lo_65536x8192": Workload("gemv16x12_bf16lo_65536x8192", 16, 12, 65536, 8192, 1, "f32", 2, 1000,
                                            extra={"planes": 3}),
    "gemm_bf16_32x24_131072x16384x64": Workload("gemm_bf16_32x24_131072x16384x64", 32, 24, 131072, 16384,
                                                64, "bf16", 3, 20),
    "decode64x48_16384x4096x8": Workload("decode64x48_16384x4096x8", 64, 48, 16384, 4096, 8, "f32", 4, 10000,
                                         extra={"min_parity": 8}),
    "gd20x16_262144x4096": Workload("gd20x16_262144x4096", 20, 16, 262144, 4096, 1, "f32", 5, 200,
                                    a_std=1.0 / 64.0,
                                    extra={"eta": 0.5, "noise_std": 0.1}),
    # Coded gradient descent with certified generators and one fp32 parity
    # plane: of 20000 seeded N(0,1) parity matrices per code
    # (synth.conditioned_parity_matrix(20, 16, 5, 20000, stream)), candidate
    # 19453 (code of A, stream P) and 2856 (code of A^T, stream P_T) have the
    # smallest worst decode condition numbers, 1656.6 and 1634.3 over every
    # survivor set (the plain draws: 102128 and 3518).
    "gd20x16_conditioned_262144x4096": Workload("gd20x16_conditioned_262144x4096", 20, 16, 262144, 4096, 1, "f32",
                                                5, 200, a_std=1.0 / 64.0,
                                                extra={"eta": 0.5, "noise_std": 0.1, "planes": 1,
                                                       "candidates": 20000, "parity_candidate": 19453,
                                                       "parity_candidate_T": 2856, "worst_condition": 1656.6,
                                                       "worst_condition_T": 1634.3}),
}


def gd_codes(w: Workload):
    """Parity matrices of the two codes of a coded gradient-descent workload (the
    code of A from stream P, the code of A^T from stream P_T) and the parity
    planes they are stored with: the plain seeded draws with two planes, or
    the workload's certified candidates with its plane count."""
    from .inputs import STREAM_P, STREAM_PT, conditioned_parity_matrix, parity_matrix
    if "parity_candidate" in w.extra:
        c = w.extra["candidates"]
        PA = conditioned_parity_matrix(w.n, w.k, w.seed, c, STREAM_P, pick=w.extra["parity_candidate"])[0]
        PT = conditioned_parity_matrix(w.n, w.k, w.seed, c, STREAM_PT, pick=w.extra["parity_candidate_T"])[0]
        return PA, PT, w.extra["planes"]
    return parity_matrix(w.n, w.k, w.seed), parity_matrix(w.n, w.k, w.seed, STREAM_PT), 2
