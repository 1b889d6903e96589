"""Heap maps of a plan: every tensor as a rectangle over (op, address), the
picture Section 5 and the appendix draw for each planning strategy.

Host-side export only (numpy in, text out): `rectangles` gives the
coordinates, `to_svg` and `to_csv` write them.  A tensor alive from op first
to op last inclusive occupies ops [first, last + 1) and bytes
[offset, offset + size); in a valid plan no two rectangles overlap.
"""
from __future__ import annotations

import numpy as np


def _host(a, dtype):
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(a, dtype=dtype)


def rectangles(size, first, last, offset) -> np.ndarray:
    """int64[n, 4]: (op_begin, op_end, byte_begin, byte_end) per tensor."""
    size, offset = _host(size, np.int64), _host(offset, np.int64)
    first, last = _host(first, np.int64), _host(last, np.int64)
    if not (size.shape == first.shape == last.shape == offset.shape):
        raise ValueError("inconsistent array lengths")
    return np.stack([first, last + 1, offset, offset + size], axis=1)


def to_csv(size, first, last, offset) -> str:
    r = rectangles(size, first, last, offset)
    lines = ["id,op_begin,op_end,byte_begin,byte_end"]
    lines += [f"{i},{a},{b},{c},{d}" for i, (a, b, c, d) in enumerate(r.tolist())]
    return "\n".join(lines) + "\n"


def to_svg(size, first, last, offset, *, width: int = 800, height: int = 400,
           title: str | None = None) -> str:
    """An SVG drawing: ops along x, addresses up along y, one rectangle per
    tensor (colour from its id), the plan's peak as the top edge."""
    r = rectangles(size, first, last, offset).astype(np.float64)
    ops = max(float(r[:, 1].max()) if len(r) else 1.0, 1.0)
    peak = max(float(r[:, 3].max()) if len(r) else 1.0, 1.0)
    sx, sy = width / ops, height / peak
    out = [f'<svg xmlns="http://www.w3.org/2000/svg" width="{width}" height="{height + 20}" '
           f'viewBox="0 0 {width} {height + 20}">']
    if title:
        out.append(f'<title>{title}</title>')
    out.append(f'<rect x="0" y="0" width="{width}" height="{height}" fill="white" '
               f'stroke="black" class="frame"/>')
    for i, (a, b, c, d) in enumerate(r.tolist()):
        hue = (i * 137.508) % 360.0
        out.append(f'<rect class="tensor" data-id="{i}" x="{a * sx:.3f}" '
                   f'y="{height - d * sy:.3f}" width="{(b - a) * sx:.3f}" '
                   f'height="{(d - c) * sy:.3f}" fill="hsl({hue:.1f},60%,60%)" '
                   f'stroke="black" stroke-width="0.2"/>')
    out.append(f'<text x="2" y="{height + 15}" font-size="12">ops 0..{int(ops)}, '
               f'peak {int(peak)} bytes</text>')
    out.append("</svg>")
    return "\n".join(out) + "\n"
