"""Time every (tile, split-k) configuration of a GEMM shape on the GPU and
report the selector's choice against the fastest one.

    python -m paper_2609_16389_amd.sweep 512,4096,4096 [M,N,K ...] [--dtype bf16] [--rounds 5]

One JSON line per shape: the selected configuration, its time, the fastest
measured configuration and every configuration's median time (microseconds).
When xgemm_run cuts the call into a body and a band of C (xgemm_select_band),
that plan is timed too (key "band" in all_us) and is the selected one.
Inputs are seeded uniform[-1, 1] values generated on the device; configurations
are timed in shuffled order, several calls per timing, median over rounds.
"""
from __future__ import annotations

import argparse
import json
import random
import statistics

import torch

from . import xgemm as xg

MAX_WORKGROUPS = 4096  # configurations with more workgroups than this are skipped


def candidates(M: int, N: int, K: int, selected: tuple[int, int]):
    out = {selected}
    for tile in range(xg.XGEMM_TILE_COUNT):
        bm, bn, bk, _ = xg.xgemm_tile_info(tile)
        for split in (1, 2, 4, 8, 16):
            if split > 1 and K // split < 3 * bk:
                continue
            if -(-M // bm) * -(-N // bn) * split > MAX_WORKGROUPS:
                continue
            out.add((tile, split))
    return sorted(out)


def sweep_shape(M: int, N: int, K: int, dtype: str = "bf16", rounds: int = 5) -> dict:
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float16
    code = xg.XGEMM_BF16 if dtype == "bf16" else xg.XGEMM_FP16
    g = torch.Generator(device="cuda").manual_seed(M + N + K)
    A = (torch.rand(M, K, device="cuda", generator=g) * 2 - 1).to(tdt)
    B = (torch.rand(K, N, device="cuda", generator=g) * 2 - 1).to(tdt)
    C = torch.empty(M, N, device="cuda", dtype=torch.float32)
    h = xg.handle(torch.cuda.current_device())
    stream = torch.cuda.current_stream()
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    sel = xg.xgemm_select_config(M, N, K, code, cu)
    band = xg.xgemm_select_band(M, N, K, code, cu)
    runs = []
    if band.axis != xg.XGEMM_BAND_NONE:
        def call_band():
            rc = xg.xgemm_run(h, M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N, code, stream.cuda_stream)
            if rc != xg.XGEMM_OK:
                raise xg.XgemmError(rc)
        call_band()
        runs.append(("band", call_band))
    for tile, split in candidates(M, N, K, (sel.tile, sel.split_k)):
        cfg = xg.xgemm_config(tile=tile, split_k=split, group_m=sel.group_m, tail_split=0)

        def call(cfg=cfg):
            rc = xg.xgemm_run_config(h, M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N, code,
                                     stream.cuda_stream, cfg)
            if rc != xg.XGEMM_OK:
                raise xg.XgemmError(rc)
        call()
        runs.append(((tile, split), call))
    torch.cuda.synchronize()
    reps = max(3, min(50, int(2e8 / max(1.0, 2.0 * M * N * K / 1e3))))
    times: dict = {k: [] for k, _ in runs}
    for _ in range(rounds):
        random.shuffle(runs)
        for key, call in runs:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            call()
            e0.record(stream)
            for _ in range(reps):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            times[key].append(e0.elapsed_time(e1) / reps * 1e3)
    med = {k: statistics.median(v) for k, v in times.items()}
    best = min(med, key=med.get)
    chosen = "band" if band.axis != xg.XGEMM_BAND_NONE else (sel.tile, sel.split_k)
    name = lambda k: k if k == "band" else list(k)
    out = {"shape": [M, N, K], "dtype": dtype, "selected": name(chosen), "selected_us": round(med[chosen], 2),
           "best": name(best), "best_us": round(med[best], 2), "loss": round(med[chosen] / med[best], 3),
           "all_us": {(k if k == "band" else "%d:%d" % k): round(v, 1)
                      for k, v in sorted(med.items(), key=lambda kv: (kv[0] == "band", str(kv[0])))}}
    if band.axis != xg.XGEMM_BAND_NONE:
        out["band"] = {"axis": "columns" if band.axis == xg.XGEMM_BAND_COLUMNS else "rows",
                       "body_extent": band.extent, "body": [band.body.tile, band.body.split_k],
                       "band": [band.band.tile, band.band.split_k]}
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("shapes", nargs="+", help="M,N,K")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "fp16"])
    ap.add_argument("--rounds", type=int, default=5)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("sweep: needs a GPU")
    for s in args.shapes:
        M, N, K = (int(v) for v in s.split(","))
        print(json.dumps(sweep_shape(M, N, K, args.dtype, args.rounds)), flush=True)
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
