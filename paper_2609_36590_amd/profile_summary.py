#!/usr/bin/env python3
"""Summarise a rocprofv3 kernel trace (rocpd SQLite output of `rocprofv3 --kernel-trace`).

Dispatches are grouped by kernel and launch shape (grid, workgroup, dynamic LDS), so that the
same kernel template launched for different passes (prefill, verify, draft) is listed apart.

usage: python3 paper_2609_36590_amd/profile_summary.py <run_results.db> [--min-calls N] [name-substring ...]
       python3 paper_2609_36590_amd/profile_summary.py --pmc <run_results.db> [--min-calls N] [name-substring ...]

With --pmc the database comes from a `rocprofv3 --pmc <counter>` run and the table lists, per
kernel and launch shape, the mean value of each collected counter per dispatch.

       python3 paper_2609_36590_amd/profile_summary.py --traffic <dir> <kernel> <name-substring> <grid> <lds> <out.md>

       python3 paper_2609_36590_amd/profile_summary.py --step-traffic <dir> <out.md>

--step-traffic writes the counted HBM bytes per decode round, verification and draft step (see
step_traffic). --traffic writes the HBM-traffic summary that bench.py reads for `roofline.traffic`, from the four runs
<dir>/pmc_copy_{FETCH,WRITE}_SIZE and <dir>/pmc_bench_{FETCH,WRITE}_SIZE (see the commands in the
written file): the dominant kernel's per-dispatch FETCH_SIZE and WRITE_SIZE, each scaled by what
the counter reads for the plain 1 GiB copy, stamped with the hash of the kernel sources.
"""
import json
import os
import sqlite3
import sys


def pmc_summary(db, filt, min_calls):
    rows = db.execute(
        "select kernel_name, grid_size, workgroup_size, lds_block_size, counter_name, count(*), avg(value), "
        "min(value), max(value) from counters_collection "
        "group by kernel_name, grid_size, workgroup_size, lds_block_size, counter_name "
        "order by avg(value) * count(*) desc").fetchall()
    print(f"{'kernel':52s} {'grid':>9s} {'wg':>5s} {'lds':>6s} {'counter':>11s} {'dispatches':>10s} "
          f"{'mean':>14s} {'min':>14s} {'max':>14s}")
    for (name, grid, wg, lds, ctr, n, avg, mn, mx) in rows:
        if n < min_calls or (filt and not any(f in name for f in filt)):
            continue
        short = name.replace("seedk::", "").replace("unsigned short", "bf16").replace("(seedk::LinArgs)", "")
        short = short.replace("(seedk::AttnArgs)", "").replace("void ", "").split("(")[0]
        print(f"{short[:52]:52s} {grid:9d} {wg:5d} {lds:6d} {ctr:>11s} {n:10d} {avg:14.2f} {mn:14.2f} {mx:14.2f}")


def counter_mean(path, name_sub, grid=None, lds=None):
    db = sqlite3.connect(path)
    q = "select avg(value), count(*) from counters_collection where kernel_name like ?"
    par = [f"%{name_sub}%"]
    if grid is not None:
        q += " and grid_size = ?"
        par.append(grid)
    if lds is not None:
        q += " and lds_block_size = ?"
        par.append(lds)
    v, n = db.execute(q, par).fetchone()
    if not n:
        raise SystemExit(f"no dispatch of '{name_sub}' (grid {grid}) in {path}")
    return v, n


COPY_BYTES = 1 << 30
COMMANDS = """```
cd /tmp && export TMPDIR=/tmp && cd <repository root>
for c in FETCH_SIZE WRITE_SIZE; do
  timeout -s KILL 120 rocprofv3 --pmc $c -d {d}/pmc_copy_$c -o run -- python3 bench.py --copy-calib
done
for c in FETCH_SIZE WRITE_SIZE; do
  timeout -s KILL 300 rocprofv3 --pmc $c -d {d}/pmc_bench_$c -o run -- python3 bench.py --profile-run --steps 20 --warmup 5
done
python3 paper_2609_36590_amd/profile_summary.py --traffic {d} {args}
```"""


def traffic(argv):
    d, kernel, name_sub, grid, lds, out = argv[0], argv[1], argv[2], int(argv[3]), int(argv[4]), argv[5]
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import bench

    run = lambda c: os.path.join(d, f"pmc_{c}", "run_results.db")
    cf, _ = counter_mean(run("copy_FETCH_SIZE"), "copyBuffer")
    cw, _ = counter_mean(run("copy_WRITE_SIZE"), "copyBuffer")
    kf, nf = counter_mean(run("bench_FETCH_SIZE"), name_sub, grid, lds)
    kw, nw = counter_mean(run("bench_WRITE_SIZE"), name_sub, grid, lds)
    rec = {"kernel": kernel, "kernel_name": name_sub, "grid_threads": grid, "lds_bytes": lds, "fetch_kib": round(kf, 3),
           "write_kib": round(kw, 3), "fetch_scale": round(COPY_BYTES / 1024 / cf, 5),
           "write_scale": round(COPY_BYTES / 1024 / cw, 5), "kernel_source_sha256": bench.kernel_source_hash()}
    tb = rec["fetch_kib"] * 1024 * rec["fetch_scale"] + rec["write_kib"] * 1024 * rec["write_scale"]
    lines = [f"# HBM traffic counters: {kernel} ({name_sub}, grid {grid} threads, {lds} B dynamic LDS)", "",
             "FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each from a rocprofv3 pass of its own, scaled",
             f"by what the same counter reads for a plain {COPY_BYTES >> 30} GiB device-to-device copy",
             f"(`__amd_rocclr_copyBuffer`): the copy reads {cf:.2f} KiB of FETCH_SIZE (scale "
             f"{rec['fetch_scale']}) and {cw:.2f} KiB of WRITE_SIZE (scale {rec['write_scale']}).", "",
             f"{kernel}: {kf:.1f} KiB fetched x {rec['fetch_scale']} + {kw:.1f} KiB written x {rec['write_scale']}"
             f" = {tb / 1e6:.2f} MB per launch (mean over {nf} / {nw} dispatches).", "",
             "Commands (one MI355X, library built by `__graft_entry__.build()`):", "",
             COMMANDS.format(d=d, args=f"{kernel} '{name_sub}' {grid} {lds} {out}"), ""]
    for c in ("copy_FETCH_SIZE", "copy_WRITE_SIZE", "bench_FETCH_SIZE", "bench_WRITE_SIZE"):
        import io
        import contextlib
        buf = io.StringIO()
        with contextlib.redirect_stdout(buf):
            pmc_summary(sqlite3.connect(run(c)), [], 1 if c.startswith("copy") else 100)
        lines += ["```", buf.getvalue().rstrip(), "```", ""]
    lines += ["Machine-readable record read by bench.py (`roofline.traffic` is reported only while the",
              "kernel sources hash to the value below):", "", "traffic-json: " + json.dumps(rec)]
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps(rec))


STEP_COMMANDS = """```
cd /tmp && export TMPDIR=/tmp && cd <repository root>
for c in FETCH_SIZE WRITE_SIZE; do
  timeout -s KILL 120 rocprofv3 --pmc $c -d {d}/pmc_copy_$c -o run -- python3 bench.py --copy-calib
  timeout -s KILL 300 rocprofv3 --pmc $c -d {d}/pmc_r10_$c -o run -- python3 bench.py --config {cfg} --k {k} --profile-run --steps 10 --warmup 5
  timeout -s KILL 300 rocprofv3 --pmc $c -d {d}/pmc_r30_$c -o run -- python3 bench.py --config {cfg} --k {k} --profile-run --steps 30 --warmup 5
  timeout -s KILL 300 rocprofv3 --pmc $c -d {d}/pmc_r10d20_$c -o run -- python3 bench.py --config {cfg} --k {k} --profile-run --steps 10 --warmup 5 --profile-drafts 20
done
python3 paper_2609_36590_amd/profile_summary.py --step-traffic {d} {out} {cfg} {k}
```"""


def group_sums(path):
    """Sum of the counter (KiB) over all dispatches, per kernel and launch shape."""
    db = sqlite3.connect(path)
    rows = db.execute("select kernel_name, grid_size, workgroup_size, lds_block_size, sum(value), count(*) "
                      "from counters_collection group by kernel_name, grid_size, workgroup_size, lds_block_size")
    return {(n, g, w, l): (v, c) for (n, g, w, l, v, c) in rows}


def step_traffic(argv):
    """HBM bytes per decode step from the counters of three profile runs that differ only in the
    number of rounds (10 vs 30) or in 20 extra draft calls: the prefill and the warm-up cancel
    in the differences. Per round = (r30 - r10) / 20, per draft step = (r10d20 - r10) / (20 k),
    per verification = per round - k draft steps."""
    d, out = argv[0], argv[1]
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import bench
    from paper_2609_36590_amd import synth

    cfg = synth.CONFIGS[argv[2]] if len(argv) > 2 else synth.C3_4B
    k = int(argv[3]) if len(argv) > 3 else 4
    run = lambda c: os.path.join(d, f"pmc_{c}", "run_results.db")
    scale = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        v, _ = counter_mean(run(f"copy_{c}"), "copyBuffer")
        scale[c] = COPY_BYTES / 1024 / v   # bytes of a copy per KiB the counter reads
    per = {}   # group -> [round bytes, draft-call bytes]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        a, b, e = group_sums(run(f"r10_{c}")), group_sums(run(f"r30_{c}")), group_sums(run(f"r10d20_{c}"))
        for key in set(a) | set(b) | set(e):
            va, vb, ve = (x.get(key, (0.0, 0))[0] for x in (a, b, e))
            r = (vb - va) / 20 * 1024 * scale[c]
            dc = (ve - va) / 20 * 1024 * scale[c]
            acc = per.setdefault(key, [0.0, 0.0])
            acc[0] += r
            acc[1] += dc
    rnd = sum(v[0] for v in per.values())
    dcall = sum(v[1] for v in per.values())
    dstep = dcall / k
    ver = rnd - k * dstep
    lens = synth.make_prompt_lengths(cfg)
    B = len(lens)
    # the runs' mean context: prompt + ~25 positions (5 warm-up and 10-30 rounds at a ~ 0)
    Ls = [n + 25 for n in lens]
    att = lambda L, layers: layers * bench.kernel_bytes(cfg, bench.binding.OP_ATTN, 0, L)
    alg_v = bench.step_bytes(cfg, B * (k + 1), Ls[0], cfg.n_layers) + sum(att(L, cfg.n_layers) for L in Ls[1:])
    alg_d = bench.step_bytes(cfg, B, Ls[0], cfg.n_dec_layers) + sum(att(L, cfg.n_dec_layers) for L in Ls[1:])
    L = int(sum(Ls) / B)
    lines = [f"# HBM traffic per decode step from rocprofv3 counters: {cfg.name}, batch {B}, k = {k}", "",
             "FETCH_SIZE and WRITE_SIZE summed over every kernel dispatch of three profile runs (prefill, 5",
             "warm-up rounds, then 10 rounds; 30 rounds; 10 rounds and 20 eager draft calls of k = 4 steps),",
             "each scaled by what the counter reads for a plain 1 GiB copy "
             f"(FETCH x {scale['FETCH_SIZE']:.5f}, WRITE x {scale['WRITE_SIZE']:.5f}). The prefill and the warm-up "
             "cancel in the differences: per round = (30 rounds - 10 rounds) / 20, per draft step = (extra",
             "draft calls) / (20 k), per verification = per round - k draft steps. Algorithmic bytes at the",
             f"runs' mean context (~{L} positions): verification {alg_v / 1e9:.4f} GB, draft step {alg_d / 1e9:.4f} GB.",
             "", "| | counted HBM bytes | algorithmic bytes | counted / algorithmic |", "|---|---|---|---|",
             f"| round (k draft steps + verification) | {rnd / 1e9:.4f} GB | {(alg_v + k * alg_d) / 1e9:.4f} GB | "
             f"{rnd / (alg_v + k * alg_d):.3f} |",
             f"| verification | {ver / 1e9:.4f} GB | {alg_v / 1e9:.4f} GB | {ver / alg_v:.3f} |",
             f"| draft step | {dstep / 1e9:.4f} GB | {alg_d / 1e9:.4f} GB | {dstep / alg_d:.3f} |", "",
             "Per kernel and launch shape (MB per round; MB per draft call of k steps):", "", "```",
             f"{'kernel':60s} {'grid':>9s} {'wg':>5s} {'lds':>6s} {'MB/round':>10s} {'MB/draft call':>14s}"]
    for key, (r, dc) in sorted(per.items(), key=lambda kv: -kv[1][0]):
        if abs(r) < 0.05e6 and abs(dc) < 0.05e6:
            continue
        name = key[0].replace("seedk::", "").replace("unsigned short", "bf16").replace("void ", "")
        name = name.replace("(seedk::LinArgs)", "").replace("(seedk::AttnArgs)", "").split("(")[0]
        lines.append(f"{name[:60]:60s} {key[1]:9d} {key[2]:5d} {key[3]:6d} {r / 1e6:10.2f} {dc / 1e6:14.2f}")
    lines += ["```", "", "Commands (one MI355X, library built by `__graft_entry__.build()`):", "",
              STEP_COMMANDS.format(out=out, d=d, cfg=cfg.name, k=k), ""]
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(json.dumps({"round_bytes": rnd, "verify_bytes": ver, "draft_step_bytes": dstep,
                      "alg_verify": alg_v, "alg_draft": alg_d}))


def main():
    args = sys.argv[1:]
    if args and args[0] == "--step-traffic":
        step_traffic(args[1:])
        return
    if args and args[0] == "--traffic":
        traffic(args[1:])
        return
    pmc = "--pmc" in args
    if pmc:
        args.remove("--pmc")
    min_calls = 1
    if "--min-calls" in args:
        i = args.index("--min-calls")
        min_calls = int(args[i + 1])
        del args[i:i + 2]
    db = sqlite3.connect(args[0])
    filt = args[1:]
    if pmc:
        pmc_summary(db, filt, min_calls)
        return
    rows = db.execute(
        "select name, grid_x, grid_y, grid_z, workgroup_x, lds_size, vgpr_count, accum_vgpr_count, sgpr_count, "
        "count(*), sum(duration), avg(duration), min(duration), max(duration) from kernels "
        "group by name, grid_x, grid_y, grid_z, workgroup_x, lds_size order by sum(duration) desc").fetchall()
    total = sum(r[10] for r in rows)
    print(f"{'kernel':44s} {'grid(threads)':>20s} {'wg':>5s} {'lds':>6s} {'vgpr/agpr/sgpr':>14s} "
          f"{'calls':>7s} {'total_ms':>9s} {'avg_us':>8s} {'min_us':>8s} {'max_us':>8s} {'pct':>6s}")
    for (name, gx, gy, gz, wg, lds, vg, ag, sg, n, tot, avg, mn, mx) in rows:
        if n < min_calls or (filt and not any(f in name for f in filt)):
            continue
        short = name.replace("seedk::", "").replace("unsigned short", "bf16").replace("(LinArgs)", "")
        short = short.replace("(AttnArgs)", "").replace("void ", "").split("(")[0]
        print(f"{short[:44]:44s} {f'{gx}x{gy}x{gz}':>20s} {wg:5d} {lds:6d} {f'{vg}/{ag}/{sg}':>14s} "
              f"{n:7d} {tot / 1e6:9.2f} {avg / 1e3:8.2f} {mn / 1e3:8.2f} {mx / 1e3:8.2f} {100 * tot / total:6.2f}")


if __name__ == "__main__":
    main()
