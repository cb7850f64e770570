"""Comparators that put oracle results into the library's output layouts.

Not oracle arithmetic: the oracle states what the method computes; these
helpers only rearrange its results so that the tests can compare them with
what the library writes, element by element.
"""

import numpy as np


def topk_layout(s_star, m):
    """S* laid out as the library writes topk_idx: its m highest-ranked
    members first, then the others, each part in ascending position order.
    s_star is in rank order (score descending, position ascending), as the
    oracle's topk_middle returns it.  Only the top-m subset and the whole set
    matter to the method (the dilation takes the top m as a set), so this
    layout carries everything the selection defines."""
    s_star = np.asarray(s_star, dtype=np.int64)
    return np.concatenate([np.sort(s_star[:m]), np.sort(s_star[m:])])
