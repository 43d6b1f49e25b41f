"""The oracle's lowering of a network with the product's split-K slice counts.

How many partial sums a weight gradient is split into is a blocking choice of
the device kernels; it only sizes the ``part`` variables.  The oracle's
lowering takes the counts as an input, and tests that compare the library's
function sequence or schedule with the oracle's pass in the counts the
library chose, read off the product's lowering.
"""

from oracle.lower import lower
from paper_2010_14109_amd import netdef


def lowering(spec, keep_grads=False):
    return lower(spec, keep_grads=keep_grads, slices=netdef.Net(spec, keep_grads).slices)
