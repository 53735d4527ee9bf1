"""Measurement probes behind the decode path's design (launch floor, a bare
weight stream per launch, grid barriers, the dealing of workgroups to XCDs,
workgroup-to-workgroup hand-off latency, the bf16 conversion instruction's
rounding), from libmtp_probe.so; see
csrc/probe.hip.  Prints one JSON object:

    python -m paper_2410_13839_amd.probe

Needs a GPU; the decode library does not use these kernels."""
from __future__ import annotations

import ctypes
import json
import os
import sys

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmtp_probe.so")


def _lib():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    d = ctypes.POINTER(ctypes.c_double)
    u = ctypes.POINTER(ctypes.c_uint32)
    lib.mtp_probe_launch_floor.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, d]
    lib.mtp_probe_stream.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_int, d]
    lib.mtp_probe_flag_barrier.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, d, u, u]
    lib.mtp_probe_xcc_map.argtypes = [ctypes.c_int, ctypes.c_int, u]
    lib.mtp_probe_bf16_round.argtypes = [ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
    lib.mtp_probe_handoff.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, d, u, u, u]
    return lib


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"{what} failed ({rc})")


def launch_floor(lib, grid: int, block: int, launches: int = 100) -> float:
    us = ctypes.c_double()
    _check(lib.mtp_probe_launch_floor(grid, block, launches, ctypes.byref(us)), "launch floor")
    return us.value


def stream(lib, grid: int, nbytes: int, launches: int = 12) -> float:
    us = ctypes.c_double()
    _check(lib.mtp_probe_stream(grid, nbytes, launches, ctypes.byref(us)), "stream")
    return us.value


def flag_barrier(lib, mode: int, data: bool, rounds: int = 2000):
    us, to, st = ctypes.c_double(), ctypes.c_uint32(), ctypes.c_uint32()
    _check(lib.mtp_probe_flag_barrier(mode, int(data), rounds, ctypes.byref(us), ctypes.byref(to), ctypes.byref(st)),
           "flag barrier")
    return us.value, to.value, st.value


def xcc_map(lib, grid: int, block: int) -> list[int]:
    buf = (ctypes.c_uint32 * grid)()
    _check(lib.mtp_probe_xcc_map(grid, block, buf), "xcc map")
    return list(buf)


ST_BITS = ("plain", "sc0", "sc1", "nt")
LD_BITS = ("sc0", "plain after buffer_inv sc0", "sc1", "plain after buffer_inv sc1", "nt")


def handoff(lib, st: int, ld: int, stride: int, rounds: int = 2000):
    us, to, sr, same = ctypes.c_double(), ctypes.c_uint32(), ctypes.c_uint32(), ctypes.c_uint32()
    _check(lib.mtp_probe_handoff(st, ld, stride, rounds, ctypes.byref(us), ctypes.byref(to), ctypes.byref(sr),
                                 ctypes.byref(same)), "handoff")
    return us.value, to.value, sr.value, same.value


def main() -> None:
    lib = _lib()
    out = {"launch_floor_us": {}, "stream_us": {}, "flag_barrier": {}, "xcc_map": {}, "handoff": {}}
    mism, checked = ctypes.c_uint64(), ctypes.c_uint64()
    _check(lib.mtp_probe_bf16_round(ctypes.byref(mism), ctypes.byref(checked)), "bf16 rounding")
    out["bf16_convert_vs_rne_bits"] = {"finite_floats_checked": checked.value, "mismatches": mism.value}
    print(f"[probe] bf16 conversion instruction vs RNE on the bits: {mism.value} mismatches in {checked.value}",
          file=sys.stderr, flush=True)
    # workgroup b runs on XCD (b + s) % 8, s where the previous launch's
    # dealing stopped: count the residues b % 8 whose workgroups span more
    # than one XCD (0 means b and b + 8 always share one)
    for grid, block in ((192, 1024), (384, 1024), (256, 512), (1024, 256), (257, 1024), (272, 1024)):
        ids = xcc_map(lib, grid, block)
        split = sum(1 for r in range(8) if len({x for b, x in enumerate(ids) if b % 8 == r}) > 1)
        out["xcc_map"][f"{grid}x{block}"] = {"residues_on_more_than_one_xcd": split,
                                             "rotation": (ids[0] - 0) % 8,
                                             "per_xcd": [ids.count(x) for x in range(8)]}
        print(f"[probe] xcc map {grid} x {block}: {split} residues on more than one XCD, rotation {ids[0] % 8}",
              file=sys.stderr, flush=True)
    for stride, where in ((8, "one XCD"), (1, "two XCDs")):
        for st in range(len(ST_BITS)):
            for ld in range(len(LD_BITS)):
                us, to, sr, same = handoff(lib, st, ld, stride)
                what = f"{where}: stores {ST_BITS[st]}, loads {LD_BITS[ld]}"
                out["handoff"][what] = {"us_per_handoff": round(us, 3), "timeouts": to, "stale_reads": sr,
                                        "pairs_on_one_xcd": same}
                print(f"[probe] handoff {what}: {us:.3f} us (timeouts {to}, stale {sr}, same-XCD pairs {same} of 8)",
                      file=sys.stderr, flush=True)
    for grid in (1, 64, 256, 1024):
        for block in (64, 256, 1024):
            out["launch_floor_us"][f"{grid}x{block}"] = round(launch_floor(lib, grid, block), 3)
            print(f"[probe] launch floor {grid} x {block}: {out['launch_floor_us'][f'{grid}x{block}']} us",
                  file=sys.stderr, flush=True)
    for mb in (2, 8):
        nbytes = mb << 20
        us = stream(lib, 256, nbytes)
        out["stream_us"][f"{mb}MiB_256wg"] = {"us_per_launch": round(us, 3),
                                              "GB_s": round(nbytes / (us * 1e-6) / 1e9, 1)}
        print(f"[probe] stream {mb} MiB: {us:.3f} us", file=sys.stderr, flush=True)
    for mode, data, what in ((0, False, "every workgroup polls every flag"),
                             (0, True, "every workgroup polls every flag, 256 B data each"),
                             (1, False, "workgroup 0 polls, one go word"),
                             (1, True, "workgroup 0 polls, one go word, 256 B data each")):
        us, to, st = flag_barrier(lib, mode, data)
        out["flag_barrier"][what] = {"us_per_barrier": round(us, 3), "timeouts": to, "stale_reads": st}
        print(f"[probe] barrier {what}: {us:.3f} us (timeouts {to}, stale {st})", file=sys.stderr, flush=True)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
