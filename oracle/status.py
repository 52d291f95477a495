"""Data-error bits OR-ed into the status word (same values as the library's header)."""
NAN_LOGQ = 1 << 0         # a log-probability was NaN: treated as -inf
POS_LOGQ = 1 << 1         # a log-probability was > 0: treated as 0
BAD_PARENT = 1 << 2       # parent index not in [-1, local index): treated as -1
TOO_DEEP = 1 << 3         # node depth above MAX_DEPTH: path score forced to -inf
NOT_CLOSED = 1 << 4       # a selected node's parent is not selected
OVER_CAPACITY = 1 << 5    # more selected nodes than the budget: only the first B packed
BAD_SLOT_PARENT = 1 << 6  # slot_parent not in [0, slot): slot can never be accepted
BAD_OFFSETS = 1 << 7      # malformed offsets: candidate CSR -> nothing scored or packed;
                          # slot or KV ranges -> that request's attention is skipped

MAX_DEPTH = 16
