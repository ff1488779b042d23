"""CPU oracle for the D-Quant hot path (arXiv 2609.19880).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, tables or
constants with the HIP library; it is written from the paper alone and is kept
plain and slow on purpose so that every step can be checked against the text.

Modules, in pipeline order:

* ``tables``    -- the calibration-free entropy model (Sec. 4.2 "Gaussian
                   order statistics", Sec. 4.4 sharpening, Eq. (rans) frequency
                   and cumulative tables, Alg. 1 costs r_m, Eq. (budget)).
* ``hadamard``  -- per-head Hadamard rotation (Sec. 4.2, Fig. 1).
* ``kmean``     -- windowed channel-mean removal for keys (Sec. 4.2, App. B).
* ``quantize``  -- FitMinMax, Drift (Eq. drift / lagrangian, Alg. 1), Refit,
                   FP16 metadata (Alg. 1, App. A).
* ``rans``      -- rANS encoder / decoder (Eq. rans, Alg. 2) and the fixed-size
                   record (Eq. budget, App. A).
* ``kv``        -- the whole append path over a [B, T, H, d] tensor.
* ``attention`` -- fp64 decode attention over the dequantized cache, both the
                   direct form and the folded form of Eq. (fold-key) /
                   Eq. (fold-value).
* ``fixed``     -- the fixed-width comparator at matched storage (App. B):
                   the same preprocessing, nearest-level rounding, b-bit
                   symbols in the same record size.

Readings of the paper where it is silent are listed in each module header.
"""

from . import tables, hadamard, kmean, quantize, rans, kv, attention, fixed  # noqa: F401
