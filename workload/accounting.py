"""Algorithmic work of the expert layer, used to price measured times.

FLOPs follow the paper's accounting (App. A, Eq. flops_moe): a SwiGLU expert
has three h x h_ff matrices, so one (token, expert) pair costs 6*h*h_ff FLOPs
forward (two FLOPs per multiply-add). The backward repeats the three products
twice (input gradient and weight gradient), which is the n_1 = 3 of the
policy-update time model (Sec. 7.1, Eq. layer_time_full).

Byte counts are the minimal HBM traffic of each step: every input element
read once and every output element written once.

The App. A overlap model (Eqs. flops_attn .. gpu_n_min) is reproduced here so
that its printed Qwen3-30B-A3B numbers pin the FLOP formula above.
"""
from __future__ import annotations

import math

# MI355X published peaks.
PEAK_BF16_DENSE_FLOPS = 2.5e15       # dense bf16 MFMA
PEAK_FP32_VECTOR_FLOPS = 157.3e12
PEAK_HBM_BYTES_PER_S = 8.0e12


def ffn_fwd_flops(n_pairs: int, d: int, F: int) -> float:
    """6 * n * h * h_ff: gate, up and down products over n pairs."""
    return 6.0 * n_pairs * d * F


def gate_up_flops(n_pairs: int, d: int, F: int) -> float:
    return 4.0 * n_pairs * d * F


def down_flops(n_pairs: int, d: int, F: int) -> float:
    return 2.0 * n_pairs * d * F


def permute_bytes(n_pairs: int, T: int, K: int, d: int, elem: int) -> float:
    """Read N rows of x, write N rows of x_perm, write row_to_pair, read the
    ids and write pair_to_row."""
    return 2.0 * n_pairs * d * elem + 4.0 * n_pairs + 8.0 * T * K


def combine_bytes(n_pairs: int, T: int, K: int, d: int, elem_in: int, elem_out: int) -> float:
    """Read N rows of Y_perm, write the dense [T, d] output, read the row map
    and the gates."""
    return float(n_pairs) * d * elem_in + float(T) * d * elem_out + 8.0 * T * K


def combine_bwd_bytes(n_pairs: int, T: int, K: int, d: int, elem: int) -> float:
    """Per local row: read dy[t] and Y_perm[row], write dY_perm[row]; plus the
    row map, gates and dgates."""
    return 3.0 * n_pairs * d * elem + 4.0 * n_pairs + 12.0 * T * K


def permute_bwd_bytes(n_pairs: int, T: int, K: int, d: int, elem_in: int, elem_out: int) -> float:
    return float(n_pairs) * d * elem_in + float(T) * d * elem_out + 4.0 * T * K


def wgrad_rmw_bytes(G: int, d: int, F: int, acc_elem: int = 4) -> float:
    """fp32 read-modify-write of the main-expert gradients (3 matrices)."""
    return 2.0 * G * 3 * d * F * acc_elem


def phase_bytes(N: int, g: int, T: int, K: int, d: int, F: int, b: int = 2, wgrad_group: int = 1) -> dict:
    """Algorithmic HBM bytes of every phase of one policy-update micro-step
    with N local pairs and g non-empty gradient groups (bf16 activations and
    weights of b bytes, fp32 weight gradients read and written once per
    weight-gradient launch; a launch over wgrad_group micro-steps that touch
    the same g groups shares that read-modify-write among them)."""
    r = 1.0 / wgrad_group
    return {
        "histogram_assign": 4.0 * T * K,
        "permute": permute_bytes(N, T, K, d, b),
        "gate_up_fwd": b * (N * d + g * 2 * F * d + N * F + N * 2 * F),
        "down_fwd": b * (N * F + g * d * F + N * d),
        "combine": combine_bytes(N, T, K, d, b, b),
        "combine_bwd": combine_bwd_bytes(N, T, K, d, b),
        "down_dgrad": b * (N * d + g * d * F + N * 2 * F + N * 2 * F),
        "gate_up_dgrad": b * (N * 2 * F + g * 2 * F * d + N * d),
        "gate_up_wgrad": b * (N * 2 * F + N * d) + r * 2.0 * g * 2 * F * d * 4,
        "down_wgrad": b * (N * d + N * F) + r * 2.0 * g * d * F * 4,
        "permute_bwd": permute_bwd_bytes(N, T, K, d, b, b),
    }


# --- App. A overlap model ---------------------------------------------------
def expert_bytes(h: int, h_ff: int, p: int) -> float:
    """S_e (or S_g) = 3 * h * h_ff * p bytes for a SwiGLU expert."""
    return 3.0 * h * h_ff * p


def attn_flops(n: int, h: int) -> float:
    return 8.0 * n * h * h + 2.0 * n * n * h


def moe_flops(n: int, h: int, h_ff: int, K: int, E: int) -> float:
    return 6.0 * K * n * h * h_ff + 2.0 * n * h * E


def n_min_cpu(h: int, h_ff: int, K: int, E: int, N_s: int, p_w: int, F: float, B_pcie: float) -> float:
    """Positive root of 2 n^2 + (8h + 6K h_ff + 2E) n = 3 N_s h_ff p_w F / B_pcie."""
    b = 8.0 * h + 6.0 * K * h_ff + 2.0 * E
    c = 3.0 * N_s * h_ff * p_w * F / B_pcie
    return (-b + math.sqrt(b * b + 8.0 * c)) / 4.0


def n_min_nvlink(h: int, h_ff: int, N_s: int, p_w: int, p_g: int, F: float, B_nv: float) -> float:
    """Positive root of 2 n^2 + 8 h n = 3 N_s h_ff (p_w + p_g) F / B_nv."""
    b = 8.0 * h
    c = 3.0 * N_s * h_ff * (p_w + p_g) * F / B_nv
    return (-b + math.sqrt(b * b + 8.0 * c)) / 4.0
