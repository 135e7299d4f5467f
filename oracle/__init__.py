"""Fused-3S oracle: plain, slow, obviously correct CPU reference.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP library: the arithmetic lives in ``oracle.c`` (fp64, plain
loops, its own binary16 decoder) and in the plain-Python work-list definition
below.

Functions and the passages they follow:

* :func:`attention_f64` -- Section 2.1, Eq. 1 (SDDMM -> row softmax -> SpMM)
  with the max-stabilised softmax of Section 3.5, Eq. 7; masked reading of
  the element-wise product with A (non-edges excluded from the softmax).
* :func:`bsb` -- Section 3.1, the Binary Sparse Block construction (row
  windows of 16 rows, all-zero columns removed, 16x16 blocks, one bitmap per
  block; Table 3 gives its footprint).
* :func:`attention_bf16_f64` -- the same definition on bfloat16 inputs
  (exact widening with the oracle's own bfloat16 decoder; the precision
  variant beside Table 5's fp16 scheme).
* :func:`attention_e4m3_f64` -- the same on 8-bit float (OCP e4m3) inputs,
  the low-precision inputs the paper's future work names.
* :func:`attention_bwd_f64` -- gradients of the operator (the backward pass
  the paper names as the next step): softmax Jacobian applied to dO V^T on
  the pattern, then the two products back through K and Q, and P^T dO.
* :func:`worklist` -- Section 3.2, row-window reordering (windows in
  decreasing order of block count), extended by splitting windows with more
  than ``piece`` blocks into pieces (the future-work remedy of Section 4.2).

Pins: every function is checked by ``tests/test_oracle_pins.py`` and
``tests/test_bsb_oracle.py`` against closed forms, library routines
(torch's CPU attention, scipy's softmax) and brute force; no function here is
"parity unpinned".
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = ctypes.CDLL(_build.LIB)
        i32, dbl = ctypes.c_int32, ctypes.c_double
        vp = ctypes.c_void_p
        L.oracle_half_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_half_to_double.restype = dbl
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_double.restype = dbl
        L.oracle_widen_bf16.argtypes = [ctypes.c_int64, vp, vp]
        L.oracle_widen_bf16.restype = None
        L.oracle_e4m3_to_double.argtypes = [ctypes.c_uint8]
        L.oracle_e4m3_to_double.restype = dbl
        L.oracle_widen_e4m3.argtypes = [ctypes.c_int64, vp, vp]
        L.oracle_widen_e4m3.restype = None
        L.oracle_check_csr.argtypes = [i32, vp, vp]
        L.oracle_check_csr.restype = ctypes.c_int
        L.oracle_3s_f64.argtypes = [i32, vp, vp, i32, vp, vp, vp, dbl, vp, vp, vp, i32]
        L.oracle_3s_f64.restype = ctypes.c_int
        L.oracle_3s_f64d.argtypes = [i32, vp, vp, i32, vp, vp, vp, dbl, vp, vp, vp, i32]
        L.oracle_3s_f64d.restype = ctypes.c_int
        L.oracle_3s_bwd_f64.argtypes = [i32, vp, vp, i32, vp, vp, vp, vp, dbl, vp, vp, vp]
        L.oracle_3s_bwd_f64.restype = ctypes.c_int
        L.oracle_3s_bwd_f64d.argtypes = [i32, vp, vp, i32, vp, vp, vp, vp, dbl, vp, vp, vp]
        L.oracle_3s_bwd_f64d.restype = ctypes.c_int
        L.oracle_3s_f64_rows.argtypes = [i32, vp, vp, i32, vp, vp, vp, dbl, i32, i32, vp, i32]
        L.oracle_3s_f64_rows.restype = ctypes.c_int
        L.oracle_num_windows.argtypes = [i32]
        L.oracle_num_windows.restype = i32
        L.oracle_bsb_sizes.argtypes = [i32, vp, vp, vp, vp]
        L.oracle_bsb_sizes.restype = ctypes.c_int
        L.oracle_bsb_build.argtypes = [i32, vp, vp, vp, vp, vp]
        L.oracle_bsb_build.restype = ctypes.c_int
        L.oracle_bsb_sizes_rows.argtypes = [i32, vp, vp, vp, vp, vp]
        L.oracle_bsb_sizes_rows.restype = ctypes.c_int
        L.oracle_bsb_build_rows.argtypes = [i32, vp, vp, vp, vp, vp, vp]
        L.oracle_bsb_build_rows.restype = ctypes.c_int
        _LIB = L
    return _LIB


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _csr(row_ptr, col_idx):
    rp = np.ascontiguousarray(row_ptr, dtype=np.int32)
    ci = np.ascontiguousarray(col_idx, dtype=np.int32)
    if ci.size == 0:
        ci = np.zeros(1, dtype=np.int32)  # valid pointer for an empty pattern
    return rp, ci


def _half_bits(x):
    a = np.ascontiguousarray(x)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError("expected binary16 data (float16 or uint16 bits)")
    return a


def half_to_double(bits):
    """Decode one binary16 bit pattern with the oracle's own decoder."""
    return lib().oracle_half_to_double(int(bits) & 0xFFFF)


def bf16_to_double(bits):
    """Decode one bfloat16 bit pattern with the oracle's own decoder."""
    return lib().oracle_bf16_to_double(int(bits) & 0xFFFF)


def widen_bf16(bits):
    """bfloat16 bit patterns (uint16 array) -> float64, exactly."""
    a = np.ascontiguousarray(bits)
    if a.dtype != np.uint16:
        raise TypeError("expected bfloat16 bit patterns as uint16")
    out = np.empty(a.shape, dtype=np.float64)
    lib().oracle_widen_bf16(a.size, _ptr(a), _ptr(out))
    return out


def attention_bf16_f64(row_ptr, col_idx, Q, K, V, scale, want_lse=False):
    """The operator on bfloat16 inputs (uint16 bit patterns), in fp64: the
    inputs are widened exactly and the fp64 definition is applied."""
    return attention_f64_exact(row_ptr, col_idx, widen_bf16(Q), widen_bf16(K),
                               widen_bf16(V), scale, want_lse=want_lse)


def e4m3_to_double(bits):
    """Decode one OCP e4m3 byte with the oracle's own decoder."""
    return lib().oracle_e4m3_to_double(int(bits) & 0xFF)


def widen_e4m3(bits):
    """OCP e4m3 bytes (uint8 array) -> float64, exactly."""
    a = np.ascontiguousarray(bits)
    if a.dtype != np.uint8:
        raise TypeError("expected e4m3 bytes as uint8")
    out = np.empty(a.shape, dtype=np.float64)
    lib().oracle_widen_e4m3(a.size, _ptr(a), _ptr(out))
    return out


def attention_e4m3_f64(row_ptr, col_idx, Q, K, V, scale, want_lse=False):
    """The operator on fp8 e4m3 inputs (uint8 bytes), in fp64: exact
    widening, then the fp64 definition."""
    return attention_f64_exact(row_ptr, col_idx, widen_e4m3(Q), widen_e4m3(K),
                               widen_e4m3(V), scale, want_lse=want_lse)


def check_csr(row_ptr, col_idx, N):
    rp, ci = _csr(row_ptr, col_idx)
    return lib().oracle_check_csr(int(N), _ptr(rp), _ptr(ci))


def attention_f64(row_ptr, col_idx, Q, K, V, scale, want_lse=False,
                  want_p=False, threads=0):
    """O = softmax_rows(mask_A(scale * Q K^T)) V in fp64.

    Q, K, V are N x d binary16 arrays.  Returns O (float64 N x d), plus lse
    (per row m + log l) and/or P (per CSR entry, see oracle.c) on request.
    """
    rp, ci = _csr(row_ptr, col_idx)
    q, k, v = _half_bits(Q), _half_bits(K), _half_bits(V)
    N, d = q.shape
    if k.shape != (N, d) or v.shape != (N, d):
        raise ValueError("Q, K, V must share one N x d shape")
    O = np.empty((N, d), dtype=np.float64)
    lse = np.empty(N, dtype=np.float64) if want_lse else None
    P = np.empty(max(int(rp[-1]), 1), dtype=np.float64) if want_p else None
    rc = lib().oracle_3s_f64(N, _ptr(rp), _ptr(ci), d, _ptr(q), _ptr(k), _ptr(v),
                             float(scale), _ptr(O),
                             _ptr(lse) if lse is not None else None,
                             _ptr(P) if P is not None else None, int(threads))
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    out = [O]
    if want_lse:
        out.append(lse)
    if want_p:
        out.append(P[: int(rp[-1])])
    return out[0] if len(out) == 1 else tuple(out)


def attention_f64_exact(row_ptr, col_idx, Q, K, V, scale, want_lse=False):
    """The same operator on float64 inputs (used by the finite-difference
    pins of the gradients)."""
    rp, ci = _csr(row_ptr, col_idx)
    q, k, v = (np.ascontiguousarray(x, dtype=np.float64) for x in (Q, K, V))
    N, d = q.shape
    O = np.empty((N, d), dtype=np.float64)
    lse = np.empty(N, dtype=np.float64) if want_lse else None
    rc = lib().oracle_3s_f64d(N, _ptr(rp), _ptr(ci), d, _ptr(q), _ptr(k), _ptr(v),
                              float(scale), _ptr(O),
                              _ptr(lse) if lse is not None else None, None, 0)
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    return (O, lse) if want_lse else O


def attention_bwd_f64(row_ptr, col_idx, Q, K, V, G, scale):
    """Gradients (dQ, dK, dV) of sum(O * G) for O = the 3S operator, fp64.

    Q, K, V, G are N x d arrays: binary16 (exactly widened) or float64.
    """
    rp, ci = _csr(row_ptr, col_idx)
    if np.asarray(Q).dtype == np.float64:
        arrs = [np.ascontiguousarray(x, dtype=np.float64) for x in (Q, K, V, G)]
        fn = lib().oracle_3s_bwd_f64d
    else:
        arrs = [_half_bits(x) for x in (Q, K, V, G)]
        fn = lib().oracle_3s_bwd_f64
    N, d = arrs[0].shape
    outs = [np.empty((N, d), dtype=np.float64) for _ in range(3)]
    rc = fn(N, _ptr(rp), _ptr(ci), d, *[_ptr(a) for a in arrs], float(scale),
            *[_ptr(o) for o in outs])
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    return tuple(outs)


def attention_rows_f64(row_ptr, col_idx, Q, K, V, scale, r0, r1, threads=0):
    """Rows [r0, r1) of :func:`attention_f64` (a bounded sample)."""
    rp, ci = _csr(row_ptr, col_idx)
    q, k, v = _half_bits(Q), _half_bits(K), _half_bits(V)
    N, d = q.shape
    O = np.empty((r1 - r0, d), dtype=np.float64)
    rc = lib().oracle_3s_f64_rows(N, _ptr(rp), _ptr(ci), d, _ptr(q), _ptr(k),
                                  _ptr(v), float(scale), int(r0), int(r1),
                                  _ptr(O), int(threads))
    if rc != 0:
        raise ValueError(f"oracle rejected the input (code {rc})")
    return O


def num_windows(N):
    return lib().oracle_num_windows(int(N))


def bsb(row_ptr, col_idx, N, win_row=None):
    """Binary Sparse Block layout (Section 3.1) with r = c = 16.

    ``win_row`` (T+1 ints) gives the first row of each window; by default the
    fixed windows of Algorithm 1 (16 w, the last clipped at N).  Other
    windows hold 1 to 16 consecutive rows (see :func:`segment_windows`).

    Returns a dict with ``u`` (distinct columns per window), ``nb`` (blocks
    per window), ``blk_off`` (T+1), ``cols`` (16 per block, -1 padding) and
    ``mask`` (8 uint32 words per block; bit convention in oracle.c, rows
    counted from the window's first row).
    """
    rp, ci = _csr(row_ptr, col_idx)
    if win_row is None:
        T = num_windows(N)
        wr = np.minimum(np.arange(T + 1, dtype=np.int64) * 16, N).astype(np.int32)
    else:
        wr = np.ascontiguousarray(win_row, dtype=np.int32)
        T = wr.size - 1
        if T < 0 or int(wr[-1]) != N:
            raise ValueError("win_row must end at N")
    u = np.empty(max(T, 1), dtype=np.int32)
    nb = np.empty(max(T, 1), dtype=np.int32)
    rc = lib().oracle_bsb_sizes_rows(int(T), _ptr(wr), _ptr(rp), _ptr(ci), _ptr(u),
                                     _ptr(nb))
    if rc != 0:
        raise ValueError(f"oracle bsb failed (code {rc})")
    B = int(nb[:T].sum())
    blk_off = np.empty(T + 1, dtype=np.int32)
    cols = np.empty(max(16 * B, 1), dtype=np.int32)
    mask = np.empty(max(8 * B, 1), dtype=np.uint32)
    rc = lib().oracle_bsb_build_rows(int(T), _ptr(wr), _ptr(rp), _ptr(ci),
                                     _ptr(blk_off), _ptr(cols), _ptr(mask))
    if rc != 0:
        raise ValueError(f"oracle bsb failed (code {rc})")
    return dict(u=u[:T], nb=nb[:T], blk_off=blk_off, cols=cols[: 16 * B],
                mask=mask[: 8 * B], win_row=wr)


def segment_windows(seg_ptr):
    """Row windows aligned to the graphs of a batch.

    The paper leaves the use of component boundaries in batched graphs to
    future work (Section 4.2); this is the layout used for it here.  The rows
    form consecutive segments (graph g: rows ``seg_ptr[g] .. seg_ptr[g+1]-1``)
    and a window never holds part of a segment together with rows outside it,
    except at 16-row steps inside a long segment.  Walking from row 0:

    * if more than 16 rows of the current segment remain, the window is the
      next 16 of them;
    * otherwise the window is the rest of the segment followed by every whole
      segment after it that still fits into 16 rows (empty segments always
      fit).

    Returns the windows' first rows followed by N (``T+1`` ints).
    """
    seg = [int(x) for x in seg_ptr]
    if not seg or seg[0] != 0 or any(b < a for a, b in zip(seg, seg[1:])):
        raise ValueError("seg_ptr must start at 0 and not decrease")
    N = seg[-1]
    starts = []
    r, g = 0, 0
    while r < N:
        while seg[g + 1] <= r:          # the segment that holds row r
            g += 1
        starts.append(r)
        if seg[g + 1] - r > 16:
            r += 16
            continue
        r = seg[g + 1]                  # rest of the segment ...
        g += 1
        while g + 1 < len(seg) and seg[g + 1] - starts[-1] <= 16:
            r = seg[g + 1]              # ... and the whole segments that fit
            g += 1
    starts.append(N)
    return np.array(starts, dtype=np.int32)


def worklist(nb, blk_off, piece, reorder=True):
    """Reordered work list (Section 3.2) with heavy windows split in pieces.

    Definition, in the order it is applied:

    1. Window w with ``nb[w] <= piece`` blocks is one work item covering all
       its blocks; its sort key is ``nb[w]``.
    2. A window with more blocks is split into ``np = ceil(nb/piece)`` pieces
       of whole block pairs: with ``pairs = ceil(nb/2)``, piece k covers pairs
       ``[floor(k*pairs/np), floor((k+1)*pairs/np))``.  Each piece gets a
       partial-result slot (slots numbered window by window, then piece by
       piece) and the sort key ``piece``.  Window w gets one merge record
       ``(w, first_slot, np)``.
    3. Items are listed window by window, piece by piece, then stably sorted
       by key, largest first (the paper's decreasing block count).  With
       ``reorder=False`` (the ablation without row-window reordering) the
       listing order is kept.

    Returns ``items`` (n x 4 int32: window, first block, end block, slot or
    -1) and ``merges`` (m x 3 int32).
    """
    if piece < 2 or piece % 2:
        raise ValueError("piece must be an even number >= 2")
    raw, merges = [], []
    slot = 0
    for w, n in enumerate(int(x) for x in nb):
        b0 = int(blk_off[w])
        if n <= piece:
            raw.append((n, (w, b0, b0 + n, -1)))
            continue
        npieces = -(-n // piece)
        pairs = -(-n // 2)
        merges.append((w, slot, npieces))
        for k in range(npieces):
            a = (k * pairs) // npieces
            b = ((k + 1) * pairs) // npieces
            raw.append((piece, (w, b0 + 2 * a, b0 + min(n, 2 * b), slot)))
            slot += 1
    ordered = sorted(raw, key=lambda kv: -kv[0]) if reorder else raw  # stable
    items = np.array([it for _, it in ordered], dtype=np.int32).reshape(-1, 4)
    return items, np.array(merges, dtype=np.int32).reshape(-1, 3)
