"""Oracle of endpoint selection at deployment (Alg. 2, paper Sec. 8.1) - TEST INFRASTRUCTURE ONLY.

Only `tests/` and `bench.py` may import this module; the library's own selection is C code that
shares nothing with it.

The rule, for a working set of W bytes and three endpoints (map: the kernel reads the file pages in
place; resident: one copy in device memory serves every pass; copy: the bytes are staged into
device memory for each use), given their measured rates and two residency facts:
  - a mapped set that is not resident after prefaulting lies outside the regime the selection
    covers, and the answer is "storage-bound";
  - an endpoint leaves the race when its rate is absent, when an import or capacity limit excludes
    it, and (resident only) when its allocation failed or one pass of every arm evicted the mapping;
  - each remaining endpoint costs its path time W / B;
  - map wins whenever its path time lies within the tie band theta of the fastest, since it keeps a
    single evictable copy of the bytes; otherwise the fastest endpoint wins.
The rates and residency facts are measurements and arrive here as inputs.

The paper gives no formula for the band.  The reading used here compares map's time with the
fastest remaining endpoint's, relative to the fastest: t_map - t_min <= theta * t_min.
"""
from __future__ import annotations

ENDPOINTS = ("map", "resident", "copy")


def path_time_ms(w_bytes: float, rate_bytes_per_s):
    """Path time W / B of an endpoint (Sec. 8.1), None where the rate is absent."""
    if rate_bytes_per_s is None or rate_bytes_per_s <= 0:
        return None
    return w_bytes / rate_bytes_per_s * 1e3


def select_endpoint(w_bytes: float, b_map, b_resident, b_copy, theta: float = 0.05,
                    mapped_resident: bool = True, resident_ok: bool = True, excluded=()):
    """Returns (choice, by_tie): choice in ENDPOINTS, "storage-bound" or "none"; by_tie is True
    when map was chosen by the band rather than as the outright fastest."""
    # a mapped set that is not resident: outside the regime
    if not mapped_resident:
        return "storage-bound", False
    times = {"map": path_time_ms(w_bytes, b_map), "resident": path_time_ms(w_bytes, b_resident),
             "copy": path_time_ms(w_bytes, b_copy)}
    if not resident_ok:                           # allocation failed or the mapping was evicted
        times["resident"] = None
    for e in excluded:                            # import or capacity limits
        times[e] = None
    survivors = {e: t for e, t in times.items() if t is not None}
    if not survivors:
        return "none", False
    fastest = min(survivors, key=lambda e: (survivors[e], ENDPOINTS.index(e)))
    t_min = survivors[fastest]
    if "map" in survivors and survivors["map"] - t_min <= theta * t_min:   # the tie band
        return "map", fastest != "map"
    return fastest, False
