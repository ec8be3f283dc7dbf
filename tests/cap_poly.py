"""The soft-cap polynomial table of the library (softcap_poly.h), read from
the header, and the host's rule for choosing a range from it."""
import os
import re

HDR = os.path.join(os.path.dirname(__file__), "..", "paper_2605_05023_amd", "csrc",
                   "softcap_poly.h")


def table():
    """[(R, [a0, a1, a2], rel)] widest range first, and kCapPolyMaxErr."""
    txt = open(HDR).read()
    rows = re.findall(r"\{([0-9.]+)f,\s*\{([-0-9.e]+)f,\s*([-0-9.e]+)f,\s*([-0-9.e]+)f\},\s*"
                      r"([0-9.e-]+)\}", txt)
    fits = [(float(r), [float(a0), float(a1), float(a2)], float(e)) for r, a0, a1, a2, e in rows]
    max_err = float(re.search(r"kCapPolyMaxErr = ([0-9.e-]+);", txt).group(1))
    return fits, max_err


def choose(cu):
    """The host's choice (attn_api.cpp) for a cap of cu score units: the
    widest range R with cu * R * rel within kCapPolyMaxErr."""
    fits, max_err = table()
    for r, a, e in fits:
        if cu * r * e <= max_err:
            return r, a, e
    return fits[-1]


def cap_poly_range(cu):
    return choose(cu)[0]
