#!/usr/bin/env python3
"""Benchmark of the provenance-bound key path on one MI355X.

One step = one pass of the whole hot path over one synthetic request batch, inputs resident in
HBM: key offsets -> descriptor digests -> chained block keys -> longest-prefix lookup -> store of
the misses (then the step's new entries are rolled back so that every step meets the same
index).  Consecutive steps run on two streams: the derive of step k+1 overlaps the index work of
step k, which stays in step order on its own stream.  A serial run of the same steps is reported
beside it.  The default workload is the largest configuration: 16384 requests x 4096 tokens, block
16, 20 registered dimensions, probing a 2^26-slot index that holds 2^25 entries (load 0.5).

Prints one JSON line: Gkeys/s (keys derived and probed per second), the derive kernel's share of
the int32 VALU roofline, the lookup's and the store's share of HBM bandwidth, and the CPU oracle
timed on the host cores.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X: 256 CUs x 4 SIMD16 = 64 int32 lanes per clock per CU, 2.4 GHz peak engine clock.
CUS, LANES_PER_CU, CLOCK_HZ = 256, 64, 2.4e9
INT_PEAK = CUS * LANES_PER_CU * CLOCK_HZ                  # 39.3 T int32 lane-ops/s
OPS_PER_COMPRESSION = 1384                                # minimal gfx950 VALU lane-ops per SHA-256 block
HBM_PEAK_GBS = 8000.0

WORKLOAD_TEXT = {
    "tiny": "8 req x 256 tok, block 16, 1K-slot index",
    "c2": "1024 req x 2048 tok (64 shared prefixes), vocab 128256, block 16, 32 provenance classes, "
          "4M-slot index at load 0.5",
    "c3": "4096 req x 8192 tok, chunk 256, Zipf(1.1) over 512 prefixes, 16 descriptors, 512K-slot index",
    "c4": "16384 req x 4096 tok, block 16, 20 dimensions, 64M-slot index with 2^25 entries",
    "c5": "256 req x 131072 tok, block 16, groups of 4 with uniform fork points, 4M-slot index",
    "omission": "differential omission test (Eq. 4): 512 req x 1024 tok, block 16, 20 registered dimensions, "
                "22 bindings (complete, 20 leave-one-out, token-only) x (base + 20 one-dimension variants)",
    "identity-adapter": "content identity of a LoRA adapter: 392 bfloat16 tensors (rank 8, 28 layers x 7 "
                        "projections of a 7B-class model), 36.7 MB",
    "identity-checkpoint": "content identity of a 0.5 B-parameter checkpoint: 290 bfloat16 tensors (24 layers, "
                           "hidden 896, vocabulary 151936), 988 MB",
    "budget": "fixed-budget tier: stream of 1024 req x 2048 tok batches (64 shared prefixes, fresh suffixes), "
              "block 16, provenance classes drawn uniformly, 1M-slot index with a 2^18-entry budget; each step "
              "touching lookup, touching store, generational eviction",
}


DERIVE_SOURCES = ["paper_2609_38706_amd/csrc/k_derive.hip", "paper_2609_38706_amd/csrc/pkv_internal.h"]
TABLE_SOURCES = ["paper_2609_38706_amd/csrc/k_table.hip", "paper_2609_38706_amd/csrc/pkv_internal.h"]
HBM_PEAK = 8.0e12             # MI355X HBM3E, bytes/s
EVENT_STRIDE = 10             # derive launches of the timed region between two timed ones
BYTES_PER_PROBE = 80          # the key bytes of one 4-slot bucket (64) + the 16-byte probe key
# One insert of the store path: the 64 key bytes of the home bucket read, an 8-byte compare-and-swap,
# the 16-byte key and 8-byte location written, and the 24 input bytes (key + location) read.
BYTES_PER_INSERT = 120


def traffic_record(workload: str, kernel: str = "derive"):
    """The committed rocprofv3 FETCH_SIZE/WRITE_SIZE record of a kernel (derive, lookup or store) on
    a workload, or None when there is none or the kernel's source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{kernel}_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    h = hashlib.sha256()
    for f in (DERIVE_SOURCES if kernel == "derive" else TABLE_SOURCES):
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if rec.get("source_sha256") != h.hexdigest():
        return None
    return rec


def measured_traffic(workload: str, kernel: str = "derive"):
    """HBM bytes per launch from traffic_record, or None."""
    rec = traffic_record(workload, kernel)
    return None if rec is None else int(round(rec["bytes_per_launch"]))


def compressions_per_key(block: int) -> int:
    return (block + 11 + 15) // 16


# A chain's keys are strictly serial, and every SHA-256 round has a dependent path of at least four
# VALU instructions (rotate -> 3-input XOR -> sum -> sum), each about 4 cycles: one chain finishes at
# most one round per 16 cycles, whatever the kernel.  The fraction of the int32 peak that n chains
# can reach is therefore at most n x OPS_PER_COMPRESSION / (64 rounds x 16 cycles) / (lanes/clock).
DEPENDENT_OPS_PER_ROUND, CYCLES_PER_OP = 4, 4


def chain_ceiling_frac(n_chains: int) -> float:
    per_chain = OPS_PER_COMPRESSION / (64 * DEPENDENT_OPS_PER_ROUND * CYCLES_PER_OP)   # lane-ops per clock
    return min(1.0, n_chains * per_chain / (CUS * LANES_PER_CU))


# The tighter bound of the kernels' own round: one wavefront issues a VALU instruction at most every
# 4 cycles, and the lane-pair round of a chain is 10 instructions long, so a chain finishes at most
# one round per 40 cycles (and needs two lanes, so 32 chains fill a wavefront).
PAIR_ROUND_INSTRUCTIONS = 10


def issue_ceiling_frac(n_chains: int) -> float:
    per_chain = OPS_PER_COMPRESSION / (64 * PAIR_ROUND_INSTRUCTIONS * CYCLES_PER_OP)
    return min(1.0, n_chains * per_chain / (CUS * LANES_PER_CU))


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c4", choices=sorted(WORKLOAD_TEXT))
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--classes", type=int, default=8, help="provenance classes of the budget workload")
    p.add_argument("--no-saturation", action="store_true", help="skip the derive-at-full-occupancy diagnostic")
    p.add_argument("--cpu-threads", type=int, default=0,
                   help="oracle threads (0 = the CPUs this process may run on, at most the 16 a one-GPU share has)")
    p.add_argument("--calib-copy", action="store_true", help="run only a plain 1 GiB device copy (counter calibration)")
    p.add_argument("--cold-reps", type=int, default=50,
                   help="reps of the cold-cache per-kernel measurement after the timed region (0 = skip)")
    p.add_argument("--quiet", action="store_true")
    return p.parse_args()


def log(args, *a):
    if not args.quiet:
        print("[bench]", *a, file=sys.stderr, flush=True)


def calib_copy():
    import torch
    n = 1 << 30
    src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calib_copy_bytes": n}))


def setup_gpu(args, w):
    import paper_2609_38706_amd as pkv
    from paper_2609_38706_amd.pipeline import DeviceBatch
    from workloads import locations

    import torch
    table = pkv.Table(w.capacity)
    fill = None
    for pre in (w.fill, w.warmup):
        if pre is None:
            continue
        db = DeviceBatch.from_batch(pre)
        db.set_locations(locations(db.key_off.cpu().numpy(), pre.tag))
        db.digest()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        db.derive()
        ev[1].record()
        if pre is w.fill:
            torch.cuda.synchronize()
            fill = {"chains": db.n_req, "keys": db.n_keys, "block": db.block, "ms": ev[0].elapsed_time(ev[1])}
        if pre is w.warmup:
            db.lookup(table)
        else:
            db.hits.zero_()
        db.store(table)
        if db.host_status() != 0:
            raise RuntimeError(f"index preparation failed: status {db.host_status()}")
        del db
    # two buffer sets of the same batch, so that consecutive steps can overlap on two streams
    runs = []
    for _ in range(2):
        run = DeviceBatch.from_batch(w.batch)
        run.set_locations(locations(run.key_off.cpu().numpy(), w.batch.tag))
        runs.append(run)
    return pkv, table, runs, fill


def serial_leg(args, table, run):
    """Steps one after another on one stream, every kernel bracketed by events: the per-kernel times."""
    import torch
    stream = torch.cuda.current_stream()

    def step(ev=None):
        run.n_new.zero_()
        run.key_offsets()
        run.digest()
        if ev is not None:
            ev[0].record(stream)
        run.derive()
        if ev is not None:
            ev[1].record(stream)
        run.lookup(table)
        if ev is not None:
            ev[2].record(stream)
        run.store(table)
        if ev is not None:
            ev[3].record(stream)
        run.rollback(table)

    for _ in range(args.warmup):
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if run.host_status() != 0:
        raise RuntimeError(f"step failed: status {run.host_status()}")
    return {"ms": (t1 - t0) * 1e3 / args.steps,
            "derive_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs])),
            "lookup_ms": float(np.mean([e[1].elapsed_time(e[2]) for e in evs])),
            "store_ms": float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))}


def fused_leg(args, table, run):
    """The same steps on one stream with keys and hit lengths from one call (pkv_derive_lookup: the
    fused derive and lookup kernel for B = 16), the call bracketed by events.  Its hit lengths must
    equal those of the separate derive and lookup kernels (the serial pass just before)."""
    import torch
    stream = torch.cuda.current_stream()
    want = run.host_hits()

    def step(ev=None):
        run.n_new.zero_()
        run.key_offsets()
        run.digest()
        if ev is not None:
            ev[0].record(stream)
        run.derive_lookup(table)
        if ev is not None:
            ev[1].record(stream)
        run.store(table)
        run.rollback(table)

    for _ in range(args.warmup):
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if run.host_status() != 0:
        raise RuntimeError(f"fused step failed: status {run.host_status()}")
    if not (run.host_hits() == want).all():
        raise RuntimeError("fused derive-and-lookup hit lengths differ from the lookup kernel's")
    return {"ms": (t1 - t0) * 1e3 / args.steps,
            "derive_lookup_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))}


def cold_leg(args, table, run, reps):
    """Per-kernel times with cold caches, outside the timed region: before every rep (untimed) the
    index is restored from a pristine device copy and a 1 GiB scratch buffer is written, which
    evicts L2 and the 256 MB Infinity Cache; then key offsets, digests, derive, lookup and store run
    once on one stream, the last three bracketed by events.  Medians over the reps."""
    import torch
    if reps <= 0:
        return None
    pristine = table.slots.clone()
    scratch = torch.empty(1 << 28, dtype=torch.int32, device="cuda")        # 1 GiB
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]
    for i in range(reps):
        table.slots.copy_(pristine)
        scratch.fill_(i)
        run.n_new.zero_()
        run.key_offsets()
        run.digest()
        evs[i][0].record()
        run.derive()
        evs[i][1].record()
        run.lookup(table)
        evs[i][2].record()
        run.store(table)
        evs[i][3].record()
    torch.cuda.synchronize()
    table.slots.copy_(pristine)
    torch.cuda.synchronize()
    if run.host_status() != 0:
        raise RuntimeError(f"cold leg failed: status {run.host_status()}")
    med = lambda a, b: round(float(np.median([e[a].elapsed_time(e[b]) for e in evs])), 4)
    return {"reps": reps, "derive": med(0, 1), "lookup": med(1, 2), "store": med(2, 3),
            "how": "index restored from a pristine copy and a 1 GiB scratch buffer written before each rep"}


def gpu_leg(args, w):
    """The timed region: K steps, consecutive steps overlapped on two streams (the derive of step k+1
    runs while step k is looked up, stored and rolled back).  Only the derive is bracketed by events,
    on the stream it is launched on."""
    import torch
    from paper_2609_38706_amd.pipeline import TwoStreamRunner
    pkv, table, runs, fill = setup_gpu(args, w)
    serial = serial_leg(args, table, runs[0])
    fused = fused_leg(args, table, runs[0])
    runner = TwoStreamRunner(table)
    order = [runs[i % 2] for i in range(max(args.steps, args.warmup))]
    runner.run(order[: args.warmup], rollback=True)
    torch.cuda.synchronize()
    for r in runs:
        if r.host_status() != 0:
            raise RuntimeError(f"step failed: status {r.host_status()}")
    # every EVENT_STRIDE-th derive of the timed region is bracketed by a pair of timing events (two
    # event packets on the derive stream cost about 6 us per step, 1.5% of a c2 step)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] if i % EVENT_STRIDE == 0 else None
           for i in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runner.run(order[: args.steps], rollback=True, derive_events=evs)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for r in runs:
        if r.host_status() != 0:
            raise RuntimeError(f"step failed: status {r.host_status()}")
    run = runs[(args.steps - 1) % 2]
    hits = run.host_hits()
    nk = np.diff(run.key_off.cpu().numpy())
    probes = int(np.minimum(np.maximum(hits, 0) + 1, nk).sum())         # algorithmic: up to the first miss
    new_entries = int(run.n_new.item())
    cold = cold_leg(args, table, run, args.cold_reps)
    return {"probes": probes, "ms": (t1 - t0) * 1e3 / args.steps, "derive_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs if e is not None])),
            "derive_timed_launches": sum(e is not None for e in evs), "serial": serial, "fused": fused, "n_keys": run.n_keys, "n_req": run.n_req, "hit_blocks": int(hits.sum()),
            "new_entries": new_entries, "fill": fill, "cold": cold}


def saturation_leg(args, n_chains=131072, blocks=16, reps=5):
    """Derive alone on a batch with enough chains to fill every SIMD (131072 chains x 16 keys, B=16,
    random tokens): the one shape where the int32 VALU peak is reachable.  A diagnostic, not the
    headline value."""
    import torch
    from paper_2609_38706_amd.pipeline import DeviceBatch
    rng = np.random.default_rng(0x5EED0006)
    tokens = rng.integers(0, 128256, size=n_chains * blocks * 16, dtype=np.int32)
    off = np.arange(n_chains + 1, dtype=np.int64) * (blocks * 16)
    descs = [[(b"model_id", b"saturation"), (b"salt", bytes([i]) * 8)] for i in range(16)]
    db = DeviceBatch(tokens, off, 16, descs, (np.arange(n_chains) % 16).astype(np.int32))
    db.digest()
    db.derive()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        db.derive()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    ops = db.n_keys * compressions_per_key(16) * OPS_PER_COMPRESSION
    return {"chains": n_chains, "keys": db.n_keys, "derive_ms": round(ms, 4),
            "gkeys_per_s": round(db.n_keys / (ms * 1e-3) / 1e9, 4),
            "achieved": round(ops / (ms * 1e-3) / 1e12, 4), "peak": round(INT_PEAK / 1e12, 4), "unit": "Tops/s",
            "frac": round(ops / (ms * 1e-3) / INT_PEAK, 4)}


def omission_leg(args):
    """Key-level differential omission test: every (binding, dimension) variant of a 20-dimension
    registry derived in one launch, base keys stored, variant keys looked up, hits summed."""
    import torch
    from paper_2609_38706_amd.omission import OmissionRun
    from workloads import make_omission
    case = make_omission()
    run = OmissionRun(case)
    for _ in range(args.warmup):
        run.run()
    torch.cuda.synchronize()
    res = run.result()
    expect = np.array([[0 if (names is None or d in names) else res["blocks"] for d in case.dims]
                       for _label, names in case.bindings])
    if not (res["collisions"] == expect).all():
        raise RuntimeError("omission test: collision matrix differs from its closed form")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        run.run(derive_events=evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    run.result()
    return {"ms": (t1 - t0) * 1e3 / args.steps, "derive_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs])),
            "n_keys": run.n_keys, "n_req": run.db.n_req, "block": case.batch.block, "case": case,
            "omissions": int(res["omission"].sum())}


def tree_compressions(nbytes):
    """SHA-256 compressions of one tensor's tree (leaves of 1024 bytes with a prefix byte, nodes of up
    to 16 digests with a prefix byte)."""
    blocks = lambda m: (m + 9 + 63) // 64
    if nbytes == 0:
        return 1
    full, last = divmod(nbytes, 1024)
    counts = [1024] * full + ([last] if last else [])
    total = sum(blocks(1 + c) for c in counts)
    n = len(counts)
    while n > 1:
        groups = [min(16, n - i) for i in range(0, n, 16)]
        total += sum(blocks(1 + 32 * k) for k in groups)
        n = len(groups)
    return total


def identity_leg(args, kind):
    import torch
    from paper_2609_38706_amd.identity import TensorPool, content_identity
    from workloads import identity_shapes
    shapes = identity_shapes(kind)
    g = torch.Generator(device="cuda").manual_seed(0x5EED000A)
    tensors = [torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16) for _, _, shape in shapes]
    pool = TensorPool(tensors)
    nbytes = sum(pool.nbytes)
    comps = sum(tree_compressions(n) for n in pool.nbytes)
    for _ in range(args.warmup):
        pool.compute_roots()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for e in evs:
        e[0].record()
        pool.compute_roots()
        e[1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    pool.host_roots()
    t2 = time.perf_counter()
    ident = content_identity([(n, t) for (n, _, _), t in zip(shapes, tensors)])
    t3 = time.perf_counter()
    return {"ms": (t1 - t0) * 1e3 / args.steps, "pass_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs])),
            "identity_ms": (t3 - t2) * 1e3, "nbytes": nbytes, "compressions": comps, "identity": ident.hex(),
            "tensors": [(n, dt, sh, t) for (n, dt, sh), t in zip(shapes, tensors)]}


def identity_cpu_leg(args, g, target_s=10.0):
    """The oracle's identity of the same bytes, repeated until about `target_s` seconds."""
    from oracle.identity import identity as oracle_identity
    ts = [(n, dt, sh, t.contiguous().view(-1).view(__import__("torch").uint8).cpu().numpy().tobytes())
          for n, dt, sh, t in g["tensors"]]
    total, reps, ident = 0.0, 0, None
    while total < target_s:
        t0 = time.perf_counter()
        ident = oracle_identity(ts)
        total += time.perf_counter() - t0
        reps += 1
    if ident.hex() != g["identity"]:
        raise RuntimeError("identity: GPU and oracle disagree")
    return {"value": round(reps * g["nbytes"] / total / 1e9, 6), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} identities of the same {g['nbytes'] / 1e6:.1f} MB (plain tree walk, one SHA-256 per "
                      f"leaf and node, single thread); {total:.2f} s", "seconds": round(total, 3), "steps": reps}


def budget_leg(args):
    """Steps of a fixed-budget tier over a cyclic stream of batches: derive, touching lookup,
    touching store, eviction to the budget.  Retention = hit blocks / prefix blocks requested."""
    import torch
    import paper_2609_38706_amd as pkv
    from paper_2609_38706_amd.pipeline import DeviceBatch, TwoStreamRunner
    from workloads import locations, make_budget
    batches, cap, budget = make_budget(classes=args.classes)
    table = pkv.Table(cap, epochs=True)
    dbs = []
    for b in batches:
        db = DeviceBatch.from_batch(b)
        db.set_locations(locations(db.key_off.cpu().numpy(), b.tag))
        dbs.append(db)
    n_ev = torch.zeros(1, dtype=torch.int64, device="cuda")
    runner = TwoStreamRunner(table)
    state = {"epoch": 0}

    def index_work(marks=None, hits_out=None, ev_out=None):
        """Touching lookup, touching store and eviction of one step; epochs advance in step order."""
        def work(k, db, s):
            state["epoch"] += 1
            e = state["epoch"]
            if marks is not None:
                marks[k][0].record(s)
            with torch.cuda.stream(s):
                db.n_new.zero_()
            pkv.pkv_lookup_prefix_touch(table, db.keys, db.key_off, e, db.hits[: db.n_req], db.status, s)
            pkv.pkv_store_touch(table, db.keys, db.key_off, db.hits[: db.n_req], db.locs, db.n_new, db.status, e,
                                stream=s)
            if marks is not None:
                marks[k][1].record(s)
            pkv.pkv_table_evict(table, budget, n_ev, s)
            if marks is not None:
                marks[k][2].record(s)
            if hits_out is not None:
                with torch.cuda.stream(s):
                    hits_out[k].copy_(db.hits[: db.n_req])
                    ev_out[k:k + 1].copy_(n_ev)
        return work

    first = max(args.warmup, 2 * len(dbs))
    runner.run([dbs[i % len(dbs)] for i in range(first)], index_work=index_work())
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    hits = torch.zeros((args.steps, dbs[0].n_req), dtype=torch.int32, device="cuda")
    evicted = torch.zeros(args.steps, dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runner.run([dbs[(first + k) % len(dbs)] for k in range(args.steps)], derive_events=evs,
               index_work=index_work(marks, hits, evicted))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for db in dbs:
        if db.host_status() != 0:
            raise RuntimeError(f"budget step failed: status {db.host_status()}")
    h = hits.cpu().numpy()
    pre = np.stack([batches[(first + k) % len(batches)].meta["prefix_blocks"] for k in range(args.steps)])
    if (h > pre).any():
        raise RuntimeError("budget tier: a request hit beyond its shared prefix")
    n_keys = sum(dbs[(first + k) % len(dbs)].n_keys for k in range(args.steps))
    return {"ms": (t1 - t0) * 1e3 / args.steps, "n_keys_per_step": n_keys // args.steps,
            "derive_ms": float(np.mean([e[0].elapsed_time(e[1]) for e in evs])),
            "index_ms": float(np.mean([m[0].elapsed_time(m[1]) for m in marks])),
            "evict_ms": float(np.mean([m[1].elapsed_time(m[2]) for m in marks])),
            "retention": float(h.sum() / pre.sum()), "evicted_per_step": float(evicted.float().mean().item()),
            "n_req": dbs[0].n_req, "capacity": cap, "budget": budget, "batches": batches, "first": first}


def budget_cpu_leg(args, g, target_s=10.0):
    """The oracle on the same step sequence (touching lookup, touching store, eviction), from an
    empty index, until about `target_s` seconds; rate in keys per second."""
    import oracle
    from workloads import locations
    threads, _host = cpu_threads(args)
    batches = g["batches"]
    idx = oracle.Index(g["capacity"])
    total, keys_done, i = 0.0, 0, 0
    while total < target_s:
        b = batches[i % len(batches)]
        i += 1
        t0 = time.perf_counter()
        ko = oracle.key_offsets(b.tok_off, b.block)
        keys = oracle.derive(b.tokens, b.tok_off, oracle.batch_digests(b), b.block, threads)
        hits = idx.lookup_touch(keys, ko, i)
        assert idx.store_touch(keys, ko, hits, locations(ko, b.tag), i) == 0
        idx.evict(g["budget"])
        total += time.perf_counter() - t0
        keys_done += int(ko[-1])
    return {"value": round(keys_done / total / 1e9, 6), "unit": "Gkeys/s", "cores": threads, "kind": "oracle",
            "sample": f"{i} steps of the same batch stream from an empty index (digests, derive on {threads} threads, "
                      f"touching lookup and store and eviction single-threaded); {total:.2f} s",
            "seconds": round(total, 3), "steps": i}


def omission_cpu_leg(args, case, n_keys, target_s=10.0):
    """The oracle's omission matrix on the same case, repeated until about `target_s` seconds."""
    from oracle.omission import omission_matrix
    threads, _host = cpu_threads(args)
    total, reps = 0.0, 0
    while total < target_s:
        t0 = time.perf_counter()
        omission_matrix(case, threads)
        total += time.perf_counter() - t0
        reps += 1
    return {"value": round(reps * n_keys / total / 1e9, 6), "unit": "Gkeys/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full omission tests ({len(case.bindings)} bindings x {len(case.dims)} dimensions over "
                      f"{case.batch.n_req} requests; the oracle derives both configurations of every pair and "
                      f"compares keys position by position, derive on {threads} threads); {total:.2f} s; rate in "
                      f"the test's own {n_keys} keys", "seconds": round(total, 3), "steps": reps}


def cpu_leg(args, w, target_s=10.0, max_reps=2000):
    """The oracle as it stands, on the host cores: full steps of the same workload, each on a fresh
    copy of the prepared index, repeated until about `target_s` seconds of timed CPU work.  Derive,
    lookup (read-only) and the store's sort run on the same threads; the store's merge and the
    descriptor digests on one."""
    import oracle
    from workloads import locations
    threads, host = cpu_threads(args)
    idx = oracle.Index(w.capacity, threads=threads)
    for pre in (w.fill, w.warmup):
        if pre is None:
            continue
        ko = oracle.key_offsets(pre.tok_off, pre.block)
        keys = oracle.derive(pre.tokens, pre.tok_off, oracle.batch_digests(pre), pre.block, threads)
        hits = idx.lookup(keys, ko) if pre is w.warmup else np.zeros(pre.n_req, np.int32)
        assert idx.store(keys, ko, hits, locations(ko, pre.tag)) == 0
        del keys
    b = w.batch
    locs = locations(oracle.key_offsets(b.tok_off, b.block), b.tag)
    total_s, total_keys, reps = 0.0, 0, 0
    phase = {"digests": 0.0, "derive": 0.0, "lookup": 0.0, "store": 0.0}
    while total_s < target_s and reps < max_reps:
        step_idx = idx.clone()                       # untimed: every step meets the same index
        t0 = time.perf_counter()
        digs = oracle.batch_digests(b)
        ko = oracle.key_offsets(b.tok_off, b.block)
        t1 = time.perf_counter()
        keys = oracle.derive(b.tokens, b.tok_off, digs, b.block, threads)
        t2 = time.perf_counter()
        hits = step_idx.lookup(keys, ko)
        t3 = time.perf_counter()
        rc = step_idx.store(keys, ko, hits, locs)
        t4 = time.perf_counter()
        assert rc == 0
        del step_idx
        for name, dt in zip(phase, (t1 - t0, t2 - t1, t3 - t2, t4 - t3)):
            phase[name] += dt
        total_s += t4 - t0
        total_keys += int(ko[-1])
        reps += 1
    n_keys = total_keys // reps
    # the derive on one thread, over the leading requests of the batch (about 2^17 keys)
    ko = oracle.key_offsets(b.tok_off, b.block)
    n_sub = max(1, min(b.n_req, int(np.searchsorted(ko, 1 << 17, side="right")) - 1))
    sub_off = np.ascontiguousarray(b.tok_off[:n_sub + 1])
    sub_tok = np.ascontiguousarray(b.tokens[:int(sub_off[-1])])
    sub_digs = np.ascontiguousarray(oracle.batch_digests(b)[:n_sub])
    t0 = time.perf_counter()
    oracle.derive(sub_tok, sub_off, sub_digs, b.block, 1)
    one_s = time.perf_counter() - t0
    return {"value": round(total_keys / total_s / 1e9, 6), "unit": "Gkeys/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full steps of the same workload ({b.n_req} requests, {n_keys} keys each), each on a "
                      f"fresh copy of the prepared index: digests, derive on {threads} threads, lookup on {threads} "
                      f"threads (read-only), store with its sort on {threads} threads; {total_s:.2f} s timed",
            "threads": threads, "host_cpus": host, "cpu_share": CPU_SHARE,
            "seconds": round(total_s, 3), "steps": reps, "cpu_model": cpu_model(),
            "phase_ms_per_step": {k: round(v / reps * 1e3, 3) for k, v in phase.items()},
            "derive_one_thread": {"requests": n_sub, "keys": int(ko[n_sub]), "seconds": round(one_s, 6),
                                  "gkeys_per_s": round(int(ko[n_sub]) / one_s / 1e9, 6)}}


# The host CPUs one GPU's share of the box comes with; the oracle uses no more threads than that.
CPU_SHARE = 16


def cpu_threads(args):
    """(threads the oracle uses, CPUs this process may run on)."""
    host = len(os.sched_getaffinity(0))
    return (args.cpu_threads or max(1, min(CPU_SHARE, host))), host


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the path is measured at its "
              f"one-GPU shape", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    if args.calib_copy:
        calib_copy()
        return
    if args.workload.startswith("identity-"):
        kind = args.workload.split("-", 1)[1]
        log(args, "content identity", kind)
        g = identity_leg(args, kind)
        ops = g["compressions"] * OPS_PER_COMPRESSION
        achieved = ops / (g["pass_ms"] * 1e-3)
        cpu = None if args.no_cpu_baseline else identity_cpu_leg(args, g)
        out = {
            "metric": "content identity throughput (GB/s of tensor bytes); % of roofline",
            "value": round(g["nbytes"] / (g["ms"] * 1e-3) / 1e9, 4), "unit": "GB/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(g["ms"], 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
            "config": {"workload": WORKLOAD_TEXT[args.workload], "name": args.workload, "bytes": g["nbytes"],
                       "tensors": len(g["tensors"]), "parallelism": "1 GPU"},
            "kernels_ms": {"roots": round(g["pass_ms"], 4), "identity_total_host": round(g["identity_ms"], 3)},
            "roofline": {"bound": "alu", "achieved": round(achieved / 1e12, 4), "peak": round(INT_PEAK / 1e12, 4),
                         "unit": "Tops/s", "frac": round(achieved / INT_PEAK, 5), "traffic": None,
                         "kernel": "tree roots", "compressions": g["compressions"]},
            "cpu_baseline": cpu,
        }
        print(json.dumps(out), flush=True)
        return
    if args.workload == "budget":
        log(args, "budget tier")
        g = budget_leg(args)
        ops = g["n_keys_per_step"] * compressions_per_key(16) * OPS_PER_COMPRESSION
        achieved = ops / (g["derive_ms"] * 1e-3)
        cpu = None if args.no_cpu_baseline else budget_cpu_leg(args, g)
        out = {
            "metric": "provenance-bound block keys derived+probed per second (Gkeys/s); % of roofline",
            "value": round(g["n_keys_per_step"] / (g["ms"] * 1e-3) / 1e9, 6), "unit": "Gkeys/s", "n_gpus": 1,
            "steps": args.steps, "warmup": max(args.warmup, 16), "ms_per_step": round(g["ms"], 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
            "config": {"workload": WORKLOAD_TEXT["budget"], "name": "budget", "classes": args.classes,
                       "requests": g["n_req"], "keys": g["n_keys_per_step"], "block": 16, "capacity": g["capacity"],
                       "budget": g["budget"], "parallelism": "1 GPU"},
            "kernels_ms": {"derive": round(g["derive_ms"], 4), "lookup+store": round(g["index_ms"], 4),
                           "evict": round(g["evict_ms"], 4)},
            "pipeline": {"streams": 2, "overlap": "derive of step k+1 with the touching lookup, touching store "
                                                  "and eviction of step k"},
            "roofline": {"bound": "alu", "achieved": round(achieved / 1e12, 4), "peak": round(INT_PEAK / 1e12, 4),
                         "unit": "Tops/s", "frac": round(achieved / INT_PEAK, 5), "traffic": None, "kernel": "derive",
                         "ops_per_key": compressions_per_key(16) * OPS_PER_COMPRESSION,
                         "chain_ceiling_frac": round(chain_ceiling_frac(g["n_req"]), 5)},
            "retention": round(g["retention"], 5), "evicted_per_step": g["evicted_per_step"],
            "cpu_baseline": cpu,
        }
        print(json.dumps(out), flush=True)
        return
    if args.workload == "omission":
        log(args, "omission test")
        g = omission_leg(args)
        ops = g["n_keys"] * compressions_per_key(g["block"]) * OPS_PER_COMPRESSION
        achieved = ops / (g["derive_ms"] * 1e-3)
        cpu = None if args.no_cpu_baseline else omission_cpu_leg(args, g["case"], g["n_keys"])
        out = {
            "metric": "provenance-bound block keys derived+probed per second (Gkeys/s); % of roofline",
            "value": round(g["n_keys"] / (g["ms"] * 1e-3) / 1e9, 6), "unit": "Gkeys/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(g["ms"], 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
            "config": {"workload": WORKLOAD_TEXT["omission"], "name": "omission", "requests": g["n_req"],
                       "keys": g["n_keys"], "block": g["block"], "parallelism": "1 GPU"},
            "kernels_ms": {"derive": round(g["derive_ms"], 4)},
            "roofline": {"bound": "alu", "achieved": round(achieved / 1e12, 4), "peak": round(INT_PEAK / 1e12, 4),
                         "unit": "Tops/s", "frac": round(achieved / INT_PEAK, 5), "traffic": None, "kernel": "derive",
                         "ops_per_key": compressions_per_key(g["block"]) * OPS_PER_COMPRESSION,
                         "chain_ceiling_frac": round(chain_ceiling_frac(g["n_req"]), 5)},
            "cpu_baseline": cpu,
            "omissions_reported": g["omissions"],
        }
        print(json.dumps(out), flush=True)
        return
    from workloads import make_workload
    log(args, "generating workload", args.workload)
    w = make_workload(args.workload)
    log(args, "gpu leg")
    g = gpu_leg(args, w)
    log(args, "gpu leg done", g)
    block = w.batch.block
    ops = g["n_keys"] * compressions_per_key(block) * OPS_PER_COMPRESSION
    achieved = ops / (g["derive_ms"] * 1e-3)
    n_chains = w.batch.n_req
    roofline = {"bound": "alu", "achieved": round(achieved / 1e12, 4), "peak": round(INT_PEAK / 1e12, 4),
                "unit": "Tops/s", "frac": round(achieved / INT_PEAK, 5), "traffic": measured_traffic(args.workload),
                "kernel": "derive", "ops_per_key": compressions_per_key(block) * OPS_PER_COMPRESSION,
                "chain_ceiling_frac": round(chain_ceiling_frac(n_chains), 5),
                "issue_ceiling_frac": round(issue_ceiling_frac(n_chains), 5)}
    ser = g["serial"]
    lookup_bps = g["probes"] * BYTES_PER_PROBE / (ser["lookup_ms"] * 1e-3)
    roofline_lookup = {"bound": "hbm", "achieved": round(lookup_bps / 1e9, 2), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                       "frac": round(lookup_bps / HBM_PEAK, 5), "traffic": measured_traffic(args.workload, "lookup"),
                       "kernel": "lookup (serial pass, events)", "probes": g["probes"],
                       "bytes_per_probe": BYTES_PER_PROBE}
    store_bps = g["new_entries"] * BYTES_PER_INSERT / (ser["store_ms"] * 1e-3)
    srec = traffic_record(args.workload, "store")
    roofline_store = {"bound": "hbm", "achieved": round(store_bps / 1e9, 2), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                      "frac": round(store_bps / HBM_PEAK, 5),
                      "traffic": None if srec is None else int(round(srec["bytes_per_launch"])),
                      "kernel": "store (k_store; serial pass, events)",
                      "inserts": g["new_entries"], "bytes_per_insert": BYTES_PER_INSERT,
                      "atomics_per_insert": None if srec is None else srec.get("atomics_per_insert")}
    rates = {"derive_gkeys_per_s": round(g["n_keys"] / (g["derive_ms"] * 1e-3) / 1e9, 4),
             "lookup_gprobes_per_s": round(g["probes"] / (ser["lookup_ms"] * 1e-3) / 1e9, 4),
             "store_ginserts_per_s": round(g["new_entries"] / (ser["store_ms"] * 1e-3) / 1e9, 4)}
    fill = g["fill"]
    if fill is not None:                       # the index fill: one derive launch over many chains
        fops = fill["keys"] * compressions_per_key(fill["block"]) * OPS_PER_COMPRESSION
        fill = {"what": "derive of the index fill (untimed preparation, one launch)", "chains": fill["chains"],
                "keys": fill["keys"], "ms": round(fill["ms"], 4),
                "gkeys_per_s": round(fill["keys"] / (fill["ms"] * 1e-3) / 1e9, 4),
                "frac": round(fops / (fill["ms"] * 1e-3) / INT_PEAK, 5),
                "chain_ceiling_frac": round(chain_ceiling_frac(fill["chains"]), 5)}
    sat = None
    if not args.no_saturation:
        log(args, "saturation leg")
        sat = saturation_leg(args)
    cpu = None
    if not args.no_cpu_baseline:
        log(args, "cpu leg")
        cpu = cpu_leg(args, w)
    value = g["n_keys"] / (g["ms"] * 1e-3) / 1e9
    out = {
        "metric": "provenance-bound block keys derived+probed per second (Gkeys/s); % of roofline",
        "value": round(value, 6), "unit": "Gkeys/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(g["ms"], 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u32", "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "name": args.workload, "requests": g["n_req"],
                   "keys": g["n_keys"], "block": block, "capacity": w.capacity, "parallelism": "1 GPU"},
        "kernels_ms": {"derive": round(g["derive_ms"], 4), "lookup": round(g["serial"]["lookup_ms"], 4),
                       "store": round(g["serial"]["store_ms"], 4), "derive_serial": round(g["serial"]["derive_ms"], 4)},
        "kernels_ms_cold": g["cold"],
        "pipeline": {"streams": 2, "overlap": "derive of step k+1 with lookup/store/rollback of step k",
                     "serial_ms_per_step": round(g["serial"]["ms"], 4),
                     "serial_value": round(g["n_keys"] / (g["serial"]["ms"] * 1e-3) / 1e9, 6),
                     "hit_blocks": g["hit_blocks"], "new_entries": g["new_entries"],
                     "fused_ms_per_step": round(g["fused"]["ms"], 4),
                     "fused_derive_lookup_ms": round(g["fused"]["derive_lookup_ms"], 4),
                     "fused": "one stream: key offsets, digests, keys and hit lengths in one call "
                              "(pkv_derive_lookup), store, rollback"},
        "roofline": roofline,
        "roofline_lookup": roofline_lookup,
        "roofline_store": roofline_store,
        "rates": rates,
        "cpu_baseline": cpu,
        "derive_fill": fill,
        "derive_saturated": sat,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
