"""Byte accounting of one decode step.

``reads_dims`` is the paper's three-term read budget (arXiv 2609.03949, Sec. 3,
'The read budget, computed', Eq. (reads)): the attended tier, the index scan
(64 branch dims + r sketch dims + 1 residual scalar per archived row) and the
admitted rows.  ``step_bytes`` is the algorithmic traffic of one step of this
library on a concrete workload: what the method must move (index over archived
rows, the gathered 1152-B rows, queries and outputs), excluding intermediates
such as the key buffer.
"""
from __future__ import annotations

D_LAT, D_ROPE, D_ROW = 512, 64, 576
ROW_BYTES = 2 * D_ROW


def reads_dims(rho: float, r: int, f: float) -> float:
    """Eq. (reads): dims read per token per step."""
    return rho * D_ROW + (1.0 - rho) * (D_ROPE + r + 1) + f * D_ROW


def reads_bytes(rho: float, r: int, f: float, index_elem_bytes: int = 2) -> float:
    """Eq. (reads) in bytes: rows are 16-bit; the index at ``index_elem_bytes``."""
    return (rho * D_ROW * 2 + (1.0 - rho) * (D_ROPE + r + 1) * index_elem_bytes
            + f * D_ROW * 2)


def scan_bytes_per_row(mode: int, r: int, two_tier: bool) -> int:
    """Index bytes read per archived row by the scorer: the narrow slice
    (64 rope dims and/or r digest dims, bf16) plus, in two-tier mode, the
    three fp32 certificate scalars (eta, eps, gamma)."""
    n = (D_ROPE if mode & 1 else 0) + (r if mode & 2 else 0)
    return 2 * n + (12 if two_tier else 0)


def step_bytes(B: int, H: int, T: int, W: int, k: int, mode: int, r: int, two_tier: bool,
               admitted_total: int = 0) -> dict:
    """Algorithmic bytes of one score -> select -> [admit] -> attend step."""
    A = T - W
    scan = B * A * scan_bytes_per_row(mode, r, two_tier)
    attend = (B * (k + W) + admitted_total) * ROW_BYTES
    queries = B * H * (D_LAT + D_ROPE) * 2
    outputs = B * H * (D_LAT * 2 + 4)
    return {"scan": scan, "attend": attend, "queries": queries, "outputs": outputs,
            "total": scan + attend + queries + outputs}
