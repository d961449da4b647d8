"""Algorithmic work of the two attention phases, used for throughput and
roofline figures.

The counts follow the paper's cost analysis (Sec. 3.3, Table "tab:theory_cost"):
prefill attention with a cached prefix costs O(n*d^2 + L*n*d) and decode
O(d^2 + (r+1)*d).  Only the attention contractions (QK^T and PV) over the
visible (query, key) pairs are counted for prefill; decode counts the bytes it
must move from HBM.
"""
PAGE_SIZE = 16


def prefill_flops(hq: int, d: int, chunks) -> int:
    """Algorithmic FLOP of causal prefill attention: QK^T and PV over the
    visible (query, key) pairs only: 4*D*Hq*(n*r + n(n+1)/2) per chunk."""
    return sum(4 * d * hq * (n * r + n * (n + 1) // 2) for r, n in chunks)


def decode_bytes(hq: int, hkv: int, d: int, lens, page_size: int = PAGE_SIZE) -> int:
    """Algorithmic HBM bytes of one decode call: K and V of every visible
    token (bf16), Q and O (bf16), block-table entries and lengths."""
    lens = [int(L) for L in lens]
    kv = sum(2 * L * hkv * d * 2 for L in lens)
    qo = 2 * len(lens) * hq * d * 2
    bt = sum(4 * (-(-L // page_size)) for L in lens) + 4 * len(lens)
    return kv + qo + bt
