"""Device ceilings that bound an asynchronous SCD epoch on this GPU (measurement aid; libscdprobe.so).

    python -m paper_1702_07005_amd.ceiling [--per-xcd 262144] [--xcc-blocks 256 2048]

Prints one JSON object:
  * scattered fp32 atomic adds over the whole device into one array (the epoch's scatter);
  * the same adds into a footprint that only one XCD's workgroups touch (each workgroup adds into
    the region of the XCD it runs on, read from the hardware XCC_ID register), at agent and at
    workgroup scope, in fp32 and fp64: if an XCD's L2 resolved atomics on lines no other XCD
    touches, these would run at L2 rates;
  * the XCD each workgroup of a plain launch ran on, and the share of workgroups b that ran on
    XCD b mod 8 (the dispatch order the team kernel's placement assumes).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))

MODES = {0: "fp32_agent_device_wide", 4: "fp32_agent_xcd_local", 5: "fp32_workgroup_xcd_local",
         6: "fp64_agent_xcd_local", 7: "fp64_workgroup_xcd_local"}


def _lib():
    lib = ctypes.CDLL(os.path.join(HERE, "libscdprobe.so"))
    lib.scd_probe_rate.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)]
    lib.scd_probe_xcc_map.argtypes = [ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint32)]
    return lib


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--per-xcd", type=int, default=262_144, help="entries per XCD region (modes 4-7)")
    ap.add_argument("--device-wide", type=int, default=8 * 262_144, help="entries of the device-wide array (mode 0)")
    ap.add_argument("--xcc-blocks", type=int, nargs="*", default=[256, 2048])
    args = ap.parse_args()
    lib = _lib()
    out = {"atomic_adds_per_s": {}, "footprint_entries": {"device_wide": args.device_wide, "per_xcd": args.per_xcd}}
    for mode, name in MODES.items():
        v = ctypes.c_double()
        n = args.device_wide if mode == 0 else args.per_xcd
        rc = lib.scd_probe_rate(mode, n, None, ctypes.byref(v))
        out["atomic_adds_per_s"][name] = v.value if rc == 0 else None
        print(f"# {name}: {v.value / 1e9:.2f} G/s (rc {rc})", flush=True)
    out["xcc_map"] = {}
    for blocks in args.xcc_blocks:
        ids = (ctypes.c_uint32 * blocks)()
        rc = lib.scd_probe_xcc_map(blocks, ids)
        if rc != 0:
            out["xcc_map"][str(blocks)] = None
            continue
        got = list(ids)
        match = sum(1 for b, x in enumerate(got) if x == b % 8) / blocks
        counts = [got.count(x) for x in range(8)]
        out["xcc_map"][str(blocks)] = {"share_on_xcd_b_mod_8": match, "workgroups_per_xcd": counts,
                                       "first_16": got[:16]}
        print(f"# {blocks} workgroups: {match:.3f} on XCD b mod 8; per XCD {counts}", flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
