"""Algorithmic work of the PFC head step: the figures the roofline fractions use.

Counts what the method must do, independent of how the kernels do it
(recomputation or re-reads are not counted).  The classifier-side formulas
follow Partial FC's cost analysis: the sampled contraction costs 2*N*d*r*C
FLOPs (Eq. sampled_gemm_flops), first-order traffic per rank is
N*k*d + r*C*d/k + N*r*C elements for the class-sharded layout and
N*d + r*C*d + N*r*C for the replicated one (Eq. gemm_traffic), and a
model-parallel head holds M_W = 4*d*C/k bytes of weights and
M_logit = 4*N*C bytes of logits, M_FC ~ 3 M_W + 2 M_logit (Sec. 3.2.2).
"""

DTYPE_BYTES = {"f32": 4, "bf16": 2, "f16": 2}

# MI355X published peaks (dense): HBM3E bandwidth and MFMA throughput.
PEAK_HBM_GBPS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f16": 2500.0, "f32": 157.3}


def contraction_flops(B, d, K):
    """One of the three B x d x |S| contractions of a step (2 FLOPs per MAC)."""
    return 2 * B * d * K


def step_flops(B, d, K):
    """Forward logits + feature gradient + class gradient."""
    return 3 * contraction_flops(B, d, K)


def gather_bytes(K, d, w_dtype):
    """Reading the active class rows once (stage 3)."""
    return K * d * DTYPE_BYTES[w_dtype]


def update_bytes(K, d, w_dtype, master):
    """Compulsory traffic of the sparse update: each active row of W and of
    the fp32 momentum read and written once (and the fp32 master if kept)."""
    per_row = 2 * DTYPE_BYTES[w_dtype] + 2 * 4 + (2 * 4 if master else 0)
    return K * d * per_row


def first_order_traffic_elements(N, k, d, C, r, layout):
    """Eq. gemm_traffic (elements per rank): feature read + weight read + logit write."""
    if layout == "mp":
        return N * k * d + r * C * d / k + N * r * C
    if layout == "dp":
        return N * d + r * C * d + N * r * C
    raise ValueError(layout)


def fc_memory_bytes(N, k, d, classes_per_gpu):
    """Sec. 3.2.2: (M_W, M_logit, M_FC) in bytes of a full model-parallel fp32 head."""
    C = classes_per_gpu * k
    m_w = 4 * d * C / k
    m_logit = 4 * N * C
    return m_w, m_logit, 3 * m_w + 2 * m_logit
