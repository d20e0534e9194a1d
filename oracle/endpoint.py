"""Oracle of Alg. 2, endpoint selection at deployment (paper Sec. 8.1) - TEST INFRASTRUCTURE ONLY.

Only `tests/` and `bench.py` may import this module; the library's own selection is C code that
shares nothing with it.

The procedure, in the paper's order, for a working set W and three endpoints (map: the kernel
reads the file pages in place; resident: one copy into device memory serves every pass; copy: the
bytes are staged into device memory for each use):
  1. W is mapped and every page faulted in.
  2. A mapped set that is still not resident ends the procedure with a storage-bound verdict.
  3. B_map is measured over the whole mapped set.
  4. A resident arm is built that holds all of W.
  5. The resident endpoint leaves the race if that allocation failed or if one pass of every arm
     pushed the mapping out of memory.
  6. B_dev and B_copy are measured with the same kernel over the same set.
  7. Endpoints that break an import or capacity limit leave the race.
  8. The survivors are ordered by path time W / B; map wins whenever it is within the band theta
     (5 %) of the best, since it keeps a single evictable copy of the bytes.
  9. Otherwise the fastest survivor is the answer.
Steps 1, 3, 4 and 6 are measurements and arrive here as inputs.

Reading of step 8 (the paper gives no formula): "within theta" compares map's time with the
fastest survivor's, relative to the fastest: t_map - t_min <= theta * t_min.  Rates that are absent
(None or <= 0) count as endpoints that were not measured and are dropped with those of step 7.
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
    # step 2
    if not mapped_resident:
        return "storage-bound", False
    times = {"map": path_time_ms(w_bytes, b_map), "resident": path_time_ms(w_bytes, b_resident),
             "copy": path_time_ms(w_bytes, b_copy)}
    # step 5
    if not resident_ok:
        times["resident"] = None
    # step 7 (and endpoints without a measured rate)
    for e in excluded:
        times[e] = None
    survivors = {e: t for e, t in times.items() if t is not None}
    if not survivors:
        return "none", False
    # step 8
    fastest = min(survivors, key=lambda e: (survivors[e], ENDPOINTS.index(e)))
    t_min = survivors[fastest]
    if "map" in survivors and survivors["map"] - t_min <= theta * t_min:
        return "map", fastest != "map"
    # step 9
    return fastest, False
