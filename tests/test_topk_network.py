"""The fixed 8-input sorting network of the top-K selection (Batcher's
odd-even merge sort), read from the device header and checked on the host by
the 0-1 principle: a comparator network sorts every input iff it sorts every
0-1 input (Knuth, TAOCP vol. 3, 5.3.4).  Every one of the 2^8 binary inputs
must come out in descending order."""
import itertools
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "paper_2512_14080_amd", "csrc", "topk_net.h")


def network():
    src = open(HEADER).read()
    m = re.search(r"kNet\[(\d+)\]\[2\]\s*=\s*\{(.*?)\};", src, re.S)
    assert m, "kNet table not found"
    body = re.sub(r"//[^\n]*", "", m.group(2))
    pairs = [(int(a), int(b)) for a, b in re.findall(r"\{\s*(\d+)\s*,\s*(\d+)\s*\}", body)]
    assert len(pairs) == int(m.group(1))
    return pairs


def apply(net, v):
    v = list(v)
    for a, b in net:  # larger value to the lower index
        if v[b] > v[a]:
            v[a], v[b] = v[b], v[a]
    return v


def test_network_sorts_all_binary_inputs():
    net = network()
    assert len(net) == 19
    assert all(0 <= a < b < 8 for a, b in net)
    for bits in itertools.product((0, 1), repeat=8):
        assert apply(net, bits) == sorted(bits, reverse=True), bits


def test_network_stages():
    """Each prefix stage sorts what it claims: the first 4 comparators sort
    pairs, the first 10 sort the two halves (so the last 9 merge them)."""
    net = network()
    for bits in itertools.product((0, 1), repeat=8):
        p = apply(net[:4], bits)
        assert all(p[i] >= p[i + 1] for i in (0, 2, 4, 6))
        q = apply(net[:10], bits)
        assert q[:4] == sorted(q[:4], reverse=True) and q[4:] == sorted(q[4:], reverse=True)
