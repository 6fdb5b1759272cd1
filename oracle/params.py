"""Oracle of the parameter selection ``GetMagnusParams`` (paper Section III-D).

TEST INFRASTRUCTURE ONLY (see the package docstring).

All quantities are integers; division floors unless stated. Inputs: the
column count of C, the local-memory size s_LM in bytes and the byte sizes of
the stored types (4-byte column index, 8-byte value, 8-byte row pointer,
4-byte histogram counter, one bit of bitmap per column, load factor 1/alpha
with alpha = 2).

Readings taken where the printed formulas are garbled or under-determined
(each one reproduces every chunk count the paper prints in its two
runtime-parameter tables):

- tau: alpha*tau hash slots of (column, value) pairs fill s_LM, i.e.
  tau = s_LM / (alpha * (s_col + s_val)). The printed formula multiplies the
  two type sizes, which cannot be a byte count.
- dense width W: the largest power of two not above
  s_LM / (alpha * (s_val + s_bitmap)). Without the factor alpha the printed
  expression gives twice the widths implied by the tables.
- required chunks: ceil_pow2(C.m) / W, at least 1 (chunks must cover every
  column, so the count is rounded up, then to a power of two).
- max chunks per level: the largest power of two not above both the value of
  the local-memory equation (with one 4-byte counter per subgroup and row)
  and n_minGroupElems / (n_groupRows * 64), i.e. the mean local chunk of a
  multisplit work group keeps at least 64 elements so its writes stay
  coalesced. This gives 32 for 128 KB and 64 for 228 KB, as printed.
- levels: one level when required <= max; otherwise
  L = ceil(log2(required) / log2(max)), the first L-1 levels take `max`
  chunks and the last takes required / max^(L-1) (a ratio: the printed
  difference contradicts the hierarchy examples the paper lists).
- required == 1 (C.m <= W): no multisplit level at all.
"""
from __future__ import annotations

from dataclasses import dataclass, field

S_COL = 4
S_VAL = 8
S_ROWPTR = 8
S_HISTO = 4
ALPHA = 2
MIN_LOCAL_CHUNK = 64


def floor_pow2(x: int) -> int:
    if x < 1:
        return 0
    return 1 << (int(x).bit_length() - 1)


def ceil_pow2(x: int) -> int:
    if x <= 1:
        return 1
    return 1 << (int(x) - 1).bit_length()


@dataclass
class MagnusParams:
    tau: int
    dense_width: int
    chunks_required: int
    chunks_max: int
    min_group_elems: int
    group_rows: int
    v_chunks: list = field(default_factory=list)

    def table_string(self) -> str:
        """Formats the chunk counts the way the paper's tables print them."""
        if len(self.v_chunks) <= 1:
            return str(self.chunks_required)
        return "%d: %s" % (self.chunks_required, ", ".join(str(v) for v in self.v_chunks))


def get_magnus_params(c_m: int, s_lm: int, n_subgroups: int = 16, s_col: int = S_COL, s_val: int = S_VAL,
                      dense_width_max: int = 0, tau_max: int = 0) -> MagnusParams:
    """s_col / s_val: byte sizes of the stored column index and value (4 and
    8 unless given). dense_width_max / tau_max (0: none) cap W and tau the
    way an implementation whose accumulators hold less would; chunk counts
    then follow the capped W."""
    tau = s_lm // (ALPHA * (s_col + s_val))
    # dense accumulator: one value plus one bitmap bit per column, alpha headroom
    dense_width = floor_pow2((8 * s_lm) // (ALPHA * (8 * s_val + 1)))
    if dense_width_max:
        dense_width = min(dense_width, dense_width_max)
    chunks_required = max(1, ceil_pow2(c_m) // dense_width)
    # half of local memory holds the locally permuted elements
    min_group_elems = s_lm // (2 * (s_col + s_val))
    group_rows = -(-(min_group_elems - 1) // tau) + 1
    if tau_max:
        tau = min(tau, tau_max)
    eq = (s_lm - min_group_elems * (s_col + s_val) - S_HISTO) // (group_rows * (n_subgroups * S_HISTO + S_ROWPTR))
    chunks_max = min(floor_pow2(eq), floor_pow2(min_group_elems // (group_rows * MIN_LOCAL_CHUNK)))
    if chunks_required == 1:
        v = []
    elif chunks_required <= chunks_max:
        v = [chunks_required]
    else:
        lr = chunks_required.bit_length() - 1
        lm = chunks_max.bit_length() - 1
        levels = -(-lr // lm)
        v = [chunks_max] * (levels - 1) + [chunks_required // chunks_max ** (levels - 1)]
    return MagnusParams(tau, dense_width, chunks_required, chunks_max, min_group_elems, group_rows, v)
