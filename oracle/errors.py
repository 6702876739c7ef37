"""Error classes of the oracle (test infrastructure only).

They mirror the library's two error kinds: argument errors a caller can
check before any work (the library returns an invalid-argument status), and
faults in the data itself (the library OR-s a bit into its device error word).
"""

DERR_CONF = 1       # a confidence is NaN, negative (sign bit set) or above 1
DERR_TOKEN = 2      # a token id outside [0, vocab)
DERR_CAPACITY = 4   # a context length that leaves no room for the block


class DcutArgError(ValueError):
    """Host-checkable argument error."""


class DcutDataError(ValueError):
    """Data fault; `bits` holds the device error bits the library would set."""

    def __init__(self, bits: int, msg: str):
        super().__init__(msg)
        self.bits = bits
