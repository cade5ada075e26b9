"""Offline calibration of the latency model and its accuracy check.

The model's per-instruction costs and efficiencies (lambda and eta of Eq. 8,
the launch cost and the memory latency) are not printed in the paper; they
are obtained by profiling. This module

  * measures every legal configuration of a sample of shapes on the GPU
    (`measure`, run on the device: per-call time of back-to-back calls
    replayed from a HIP graph, operands rotating through distinct copies,
    caches flushed before every timed replay as the benchmark's other shapes
    do between its replays),
  * fits the profile constants so that the model's predictions match the
    measurements in log space (`fit`, host only), and
  * reports how well the model ranks: how often its choice is the measured
    fastest configuration (top-1) and the time lost when it is not (regret)
    (`evaluate`), for the search restricted to the taxonomy's template and
    for the open search.

    python -m paper_2608_10803_amd.calibrate measure OUT.json   (GPU)
        [--family NAME --shapes-from RECORDS.json: only that family's
        configurations, on the shapes where RECORDS.json has them]
    python -m paper_2608_10803_amd.calibrate splice OLD.json NEW.json OUT.json
        (NEW's records replace OLD's of the same family and shape)
    python -m paper_2608_10803_amd.calibrate fit RECORDS.json [--near F] [--family NAME]
        (after init on the device, so that the planner prices with the
        device's occupancies; --near F fits exactly only configurations
        within F times their shape's fastest, the others one-sided; --family
        refits only that family's configurations, the rest of the profile held)
    python -m paper_2608_10803_amd.calibrate emit FIT.json      (C++ defaults)

`fit` holds half of the measured shapes out: the profile is fitted on a
seeded half (split_shapes) and its ranking is reported on both halves, so
the held-out figures are not in-sample.
"""
import json
import math
import os
import sys
import time

import numpy as np

from . import _lib as ac

# Global profile fields fitted (log-scale multiplicative factors on the
# defaults); each kernel configuration additionally gets its own iteration and
# workgroup costs (cfg_iter, cfg_wg).
# The launch cost is not fitted: it is the measured per-kernel floor of
# back-to-back launches, and the fixed part of each configuration is in cfg_wg.
FIT_FIELDS = ["t_mem_latency", "hbm_eta", "l2_bw_cu", "unaligned_eta", "l2_hit", "swizzle_gain"]
BOUNDS = {"hbm_eta": (0.3, 1.0), "unaligned_eta": (0.3, 1.0), "l2_hit": (0.0, 0.99), "swizzle_gain": (0.5, 1.0)}
N_CFG = ac.AC_N_CFG
FLUSH_BYTES = 512 << 20


def sample_shapes(n_sweep=200, seed=11):
    """A stratified sample of the dynamic-shape sweep (evenly spaced in the
    order of the roofline floor) plus the decode-style and small-MN large-K
    shapes."""
    from workloads import gen
    sw = gen.sweep()

    def floor(s):
        M, N, K = s
        return max(2.0 * M * N * K / 2.5e15, (2.0 * M * K + 2.0 * K * N + 2.0 * M * N) / 8e12)

    order = sorted(range(len(sw)), key=lambda i: floor(sw[i]))
    pick = [sw[order[int(j)]] for j in np.linspace(0, len(sw) - 1, n_sweep)]
    return (pick + gen.skinny_m() + gen.small_mn_large_k() + write_bound_shapes() + split_k_shapes() +
            compute_bound_shapes() + tall_shapes())


def compute_bound_shapes(n=30, seed=14):
    """Shapes whose roofline floor is the MFMA one, drawn on their own: M, N,
    K log-uniform in [512, 16384], kept when the arithmetic intensity with
    bf16 output is at least 312.5 FLOP/B and M*N*K <= 2^37. They fix the
    main-loop costs of the large tiles."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        M, N, K = (int(round(math.exp(rng.uniform(math.log(512), math.log(16384))))) for _ in range(3))
        F = 2.0 * M * N * K
        Bb = 2.0 * M * K + 2.0 * K * N + 2.0 * M * N
        if F / Bb >= 312.5 and M * N * K <= 2 ** 37:
            out.append((M, N, K))
    return out


def tall_shapes(n=30, seed=16):
    """Tall-skinny shapes (A the one large operand), drawn on their own: M
    log-uniform in [1000, 100000], N uniform in 1..32, K log-uniform in
    [64, 100000] (any parity, so both load forms of the tall kernels occur),
    kept when A is at most 4 GiB. They fix the streaming kernels' costs."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        M = int(round(math.exp(rng.uniform(math.log(1000), math.log(100000)))))
        N = int(rng.integers(1, 33))
        K = int(round(math.exp(rng.uniform(math.log(64), math.log(100000)))))
        if 2.0 * M * K <= 4 * 2 ** 30:
            out.append((M, N, K))
    return out


def split_shapes(shape_keys, seed=15):
    """A seeded split of the measured shapes into a fitting half and a
    held-out half (every shape lands in exactly one)."""
    keys = sorted(shape_keys)
    perm = np.random.default_rng(seed).permutation(len(keys))
    train = {keys[i] for i in perm[: len(keys) // 2]}
    return train, set(keys) - train


def write_bound_shapes(n=50, seed=12):
    """Shapes whose traffic is mostly the output (large M x N, small K), drawn
    on their own (not from the sweep): M, N log-uniform in [2048, 100000], K
    log-uniform in [1, 400], kept when C is at least half of the bytes and
    at most 4 GiB. They fix the per-configuration write efficiency, and
    K <= 16 the small-K kernel's against the tile kernels'."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        M, N = (int(round(math.exp(rng.uniform(math.log(2048), math.log(100000))))) for _ in range(2))
        K = int(round(math.exp(rng.uniform(0.0, math.log(400)))))
        c = 2.0 * M * N
        if c >= 0.5 * (2.0 * M * K + 2.0 * K * N + c) and c <= 4 * 2 ** 30:
            out.append((M, N, K))
    return out


def split_k_shapes(n=40, seed=13):
    """Shapes with few output tiles and a long K (the split-K regime of the
    MultiCoreSplitK class), drawn on their own (not from the sweep): M, N
    log-uniform in [1, 4096], K log-uniform in [2048, 100000], kept when
    the output has fewer than 64 tiles of 32 x 32 and M*N*K <= 2^37. They
    fix how the split kernels' cost changes with the number of workgroups
    that share a CU."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        M, N = (int(round(math.exp(rng.uniform(0.0, math.log(4096))))) for _ in range(2))
        K = int(round(math.exp(rng.uniform(math.log(2048), math.log(100000)))))
        if -(-M // 32) * -(-N // 32) < 64 and M * N * K <= 2 ** 37:
            out.append((M, N, K))
    return out


def _open_profile():
    h = ac.adaptcore_get_hw()
    h.search_open = 1
    h.enable_streamk = 1
    return h


def warm_up(A, B, C, stream, seconds=2.0):
    """Keep the GPU busy with large products for a while, so that the first
    measured shapes do not run at idle clocks."""
    import torch
    n = 4096
    plan = ac.adaptcore_plan(n, n, n, ac.AC_BF16_F32OUT if C.element_size() == 4 else ac.AC_BF16_BF16OUT, 0)
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(20):
            ac.adaptcore_matmul(plan, A.data_ptr(), n, B.data_ptr(), n, C.data_ptr(), n, stream.cuda_stream)
        torch.cuda.synchronize()


def measure(out_path, shapes=None, dtype=ac.AC_BF16_BF16OUT, max_cands=100, log=print, family=None):
    """Time every legal configuration of each shape (GPU), or with `family`
    only that family's. Writes a JSON list of records {M, N, K, key, family,
    cfg fields, t}."""
    import torch
    ac.adaptcore_init()
    shapes = shapes or sample_shapes()
    base = ac.adaptcore_get_hw()
    ac.adaptcore_set_hw(_open_profile())
    dev = torch.device("cuda")
    cb = 2 if dtype == ac.AC_BF16_BF16OUT else 4
    rot = 640 << 20
    maxA = max(max(M * K for M, N, K in shapes) * 2, rot)
    maxB = max(max(K * N for M, N, K in shapes) * 2, rot)
    maxC = max(max(M * N for M, N, K in shapes) * cb, rot)
    A = torch.empty(maxA // 2, dtype=torch.bfloat16, device=dev).uniform_(-1, 1)
    B = torch.empty(maxB // 2, dtype=torch.bfloat16, device=dev).uniform_(-1, 1)
    C = torch.empty(maxC // 2, dtype=torch.bfloat16, device=dev)
    s = torch.cuda.Stream()
    ac.adaptcore_reserve_workspace(s.cuda_stream, 2 << 30)
    # read between timed replays: evicts the L2s and the 256 MB Infinity Cache,
    # so that every replay starts from the state the benchmark's replays do
    # (there, the other shapes' batches run in between)
    flush = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
    red = torch.empty(1, dtype=torch.float32, device=dev)
    warm_up(A, B, C, s)
    recs = []
    t0 = time.time()
    for si, (M, N, K) in enumerate(shapes):
        cands = ac.adaptcore_candidates(M, N, K, dtype, 0)
        if family:
            cands = [c for c in cands if c["family_name"] == family]
        if len(cands) > max_cands:
            # the model's best, every direct-to-LDS, persistent and tall configuration
            # with at most 4 splits, and a spread of the rest
            must = [i for i, c in enumerate(cands) if c["family_name"] in ("dl", "persist", "tall") and c["pk"] <= 4]
            rest = max(max_cands - 20 - len(must), 10)
            idx = sorted(set(list(range(20)) + must + list(np.linspace(20, len(cands) - 1, rest).astype(int))))
            cands = [cands[i] for i in idx]
        fa, fb, fc = 2 * M * K, 2 * K * N, cb * M * N
        for c in cands:
            plan = ac.adaptcore_plan_variant(M, N, K, dtype, 0, c["variant_key"])
            R = int(min(256, max(8, math.ceil(250e-6 / max(c["predicted_s"], 1e-6)))))

            def span(f, cap):
                f = max((f + 255) // 256 * 256, 256)
                return f, max(1, min(R, (512 << 20) // f, cap // f))
            sa, na = span(fa, maxA)
            sb, nb = span(fb, maxB)
            sc, nc = span(fc, maxC)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                for r in range(R):
                    ac.adaptcore_matmul(plan, A.data_ptr() + (r % na) * sa, max(K, 1), B.data_ptr() + (r % nb) * sb,
                                        max(N, 1), C.data_ptr() + (r % nc) * sc, max(N, 1), s.cuda_stream)
            g.replay()
            ts = []
            for _ in range(3):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.sum(flush, dim=0, keepdim=True, out=red)
                e0.record()
                g.replay()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e-3 / R)
            del g
            rec = dict(M=M, N=N, K=K, dtype=dtype, key=c["variant_key"], family=c["family_name"],
                       tile_m=c["tile_m"], tile_n=c["tile_n"], pk=c["pk"], grid=c["grid_x"] * c["grid_y"],
                       pred=c["predicted_s"], t=float(np.median(ts)))
            recs.append(rec)
        log("[%d/%d] %s %d configurations, %.0f s" % (si + 1, len(shapes), (M, N, K), len(cands), time.time() - t0))
    ac.adaptcore_set_hw(base)
    with open(out_path, "w") as f:
        json.dump(recs, f)
    return recs


def _by_shape(recs):
    out = {}
    for r in recs:
        out.setdefault((r["M"], r["N"], r["K"], r["dtype"]), {})[r["key"]] = r["t"]
    return out


def predictions(hw, shapes_keys, open_search):
    """Model predictions {shape: {key: seconds}} under profile `hw`."""
    h = hw.copy()
    h.search_open = 1 if open_search else 0
    h.enable_streamk = 1
    prev = ac.adaptcore_get_hw()
    ac.adaptcore_set_hw(h)
    out = {}
    try:
        for (M, N, K, dt) in shapes_keys:
            out[(M, N, K, dt)] = {c["variant_key"]: c["predicted_s"] for c in ac.adaptcore_candidates(M, N, K, dt, 0)}
    finally:
        ac.adaptcore_set_hw(prev)  # the caller's profile stays in force
    return out


def evaluate(recs, hw, open_search=False):
    """Top-1 agreement and regret of the model's choice against the measured
    times (only configurations that were measured are considered)."""
    meas = _by_shape(recs)
    pred = predictions(hw, list(meas), open_search)
    top1, regrets = 0, []
    for sk, mt in meas.items():
        pk = {k: v for k, v in pred[sk].items() if k in mt}
        if not pk:
            continue
        choice = min(pk, key=lambda k: (pk[k], k))
        best = min(mt.values())
        regrets.append(mt[choice] / best)
        top1 += mt[choice] <= best * 1.0000001
    r = np.array(regrets)
    return {"shapes": len(r), "top1": top1 / max(len(r), 1), "regret_geomean": float(np.exp(np.mean(np.log(r)))),
            "regret_mean": float(r.mean()), "within_10pct": float(np.mean(r <= 1.1)), "regret_max": float(r.max())}


def config_of(key):
    """Index of the calibrated cost slot of a variant key (the register-load
    form of a direct-to-LDS or tall-skinny configuration, key bit 13, has
    its own)."""
    key = int(key)
    cfg = (key >> 4) & 0xFF
    if (key & 0xF) in (ac.AC_FAMILY_DL, ac.AC_FAMILY_TALL) and (key >> 13) & 1:
        cfg |= 0x100
    return ac.adaptcore_config_index(key & 0xF, cfg)


def _log_errors(hw, meas, keys_filter=None, far=None):
    """log(predicted / measured) of every measured configuration; for the
    (shape, key) pairs in `far` only an underestimate counts (0 otherwise):
    a slow configuration must not look fast, but how slow it looks does not
    matter to the ranking."""
    pred = predictions(hw, list(meas), True)
    err = []
    for sk, mt in meas.items():
        for k, t in mt.items():
            if keys_filter is not None and k not in keys_filter:
                continue
            p = pred[sk].get(k)
            if p:
                e = math.log(p / t)
                if far is not None and (sk, k) in far:
                    e = min(e, 0.0)
                err.append(e)
    return np.array(err)


def near_records(recs, near):
    """The records whose time is within `near` times the fastest measured
    configuration of the same shape."""
    best = {}
    for r in recs:
        sk = (r["M"], r["N"], r["K"], r["dtype"])
        best[sk] = min(best.get(sk, r["t"]), r["t"])
    return [r for r in recs if r["t"] <= near * best[(r["M"], r["N"], r["K"], r["dtype"])]]


def fit(recs, hw0=None, rounds=3, iters=300, log=print, near=None, only=None):
    """Fit the profile: minimise the squared log error of the model over the
    measured configurations (with `near`, exactly only for those within that
    factor of their shape's fastest, and for the others only where the model
    underestimates them: the ranking depends on the model being right about
    the competitive candidates and on no slow one looking fast, not on how
    slow the slow ones look). Alternates a Nelder-Mead search over the global constants
    (launch, latency, bandwidth, cache hit rate) with one over the three
    constants of each kernel configuration (iteration cost, workgroup cost,
    write efficiency) on that configuration's records. With `only` (a set of
    configuration indices) the global constants and every other
    configuration are held, and one round refits those configurations alone
    (after a change to their kernels)."""
    from scipy.optimize import minimize
    hw0 = (hw0 or ac.adaptcore_get_hw()).copy()
    meas = _by_shape(recs)
    far = None
    if near:
        kept = {((r["M"], r["N"], r["K"], r["dtype"]), r["key"]) for r in near_records(recs, near)}
        far = {(sk, k) for sk, mt in meas.items() for k in mt if (sk, k) not in kept}
    by_cfg = {}
    for r in recs:
        by_cfg.setdefault(config_of(r["key"]), set()).add(r["key"])
    cur = hw0.copy()

    def loss_all(h):
        e = _log_errors(h, meas, far=far)
        return float(np.mean(np.square(e)))

    def make_global(x, base):
        h = base.copy()
        for name, v in zip(FIT_FIELDS, x):
            val = getattr(base, name) * math.exp(v)
            lo, hi = BOUNDS.get(name, (1e-12, 1e30))
            setattr(h, name, min(max(val, lo), hi))
        return h

    l0 = loss_all(cur)
    evals = 0
    for rnd in range(1 if only else rounds):
        if not only:
            base = cur.copy()
            res = minimize(lambda x: loss_all(make_global(x, base)), np.zeros(len(FIT_FIELDS)),
                           method="Nelder-Mead", options={"maxiter": iters, "xatol": 1e-3, "fatol": 1e-5})
            cur = make_global(res.x, base)
            evals += res.nfev
        for idx in sorted(by_cfg):
            if idx < 0 or (only and idx not in only):
                continue
            keys = by_cfg[idx]
            sub = {sk: mt for sk, mt in meas.items() if any(k in keys for k in mt)}

            def put(h, x):
                h.cfg_iter[idx] = math.exp(min(max(x[0], -30.0), -7.0))
                h.cfg_wg[idx] = math.exp(min(max(x[1], -30.0), -7.0))
                h.cfg_wr[idx] = math.exp(min(max(x[2], math.log(0.05)), 0.0))

            def loss_cfg(x):
                h = cur.copy()
                put(h, x)
                e = _log_errors(h, sub, keys, far=far)
                return float(np.mean(np.square(e))) if len(e) else 0.0
            if not len(_log_errors(cur, sub, keys, far=far)):
                continue  # none of this configuration's records is a candidate now
            # (an uncalibrated efficiency starts inside its range: Nelder-Mead's
            # first simplex is too small around 0 to leave the bound at 1)
            wr0 = math.log(cur.cfg_wr[idx]) if cur.cfg_wr[idx] > 0 else math.log(0.7)
            if cur.cfg_iter[idx] > 0:
                x0 = np.array([math.log(cur.cfg_iter[idx]), math.log(max(cur.cfg_wg[idx], 1e-9)), wr0])
            else:  # coarse grid for the first start
                grid = [(a, b, wr0) for a in np.log(np.logspace(-9, -5, 17)) for b in np.log([1e-8, 1e-7, 3e-7, 1e-6])]
                x0 = np.array(min(grid, key=lambda g: loss_cfg(g)))
            r2 = minimize(loss_cfg, x0, method="Nelder-Mead", options={"maxiter": 300, "xatol": 1e-3, "fatol": 1e-6})
            evals += r2.nfev
            put(cur, r2.x)
            log("  round %d configuration %d: loss %.4f" % (rnd, idx, r2.fun))
        log("fit round %d: loss %.4f" % (rnd, loss_all(cur)))
    l1 = loss_all(cur)
    log("fit: loss %.4f -> %.4f (%d evaluations)" % (l0, l1, evals))
    return cur, {"loss_before": l0, "loss_after": l1, "evals": int(evals)}


def emit_cpp(profile):
    """C++ initialisers of the fitted constants, for the library's default
    profile."""
    p = profile
    lines = ["  h.t_launch = %.4g;" % p["t_launch"], "  h.t_mem_latency = %.4g;" % p["t_mem_latency"],
             "  h.hbm_eta = %.4g;" % p["hbm_eta"], "  h.l2_bw_cu = %.4g;" % p["l2_bw_cu"],
             "  h.unaligned_eta = %.4g;" % p["unaligned_eta"], "  h.l2_hit = %.4g;" % p["l2_hit"],
             "  h.swizzle_gain = %.4g;" % p.get("swizzle_gain", 1.0)]
    it = ", ".join("%.4g" % v for v in p["cfg_iter"])
    wg = ", ".join("%.4g" % v for v in p["cfg_wg"])
    wr = ", ".join("%.4g" % v for v in p.get("cfg_wr", [0.0] * len(p["cfg_wg"])))
    lines.append("  static const double kIter[AC_N_CFG] = {%s};" % it)
    lines.append("  static const double kWg[AC_N_CFG] = {%s};" % wg)
    lines.append("  static const double kWr[AC_N_CFG] = {%s};" % wr)
    return "\n".join(lines)


def main(argv):
    fam = argv[argv.index("--family") + 1] if "--family" in argv else None
    if len(argv) >= 2 and argv[0] == "measure":
        shapes = None
        if "--shapes-from" in argv:
            with open(argv[argv.index("--shapes-from") + 1]) as f:
                old = json.load(f)
            shapes = sorted({(r["M"], r["N"], r["K"]) for r in old if fam is None or r["family"] == fam})
        measure(argv[1], shapes, family=fam)
    elif len(argv) >= 4 and argv[0] == "splice":
        # OLD NEW OUT: NEW's records replace OLD's of the same family on the same shapes
        with open(argv[1]) as f:
            old = json.load(f)
        with open(argv[2]) as f:
            new = json.load(f)
        drop = {(r["M"], r["N"], r["K"], r["dtype"], r["family"]) for r in new}
        out = [r for r in old if (r["M"], r["N"], r["K"], r["dtype"], r["family"]) not in drop] + new
        with open(argv[3], "w") as f:
            json.dump(out, f)
    elif len(argv) >= 2 and argv[0] == "fit":
        with open(argv[1]) as f:
            recs = json.load(f)
        ac.adaptcore_init()  # the device's occupancies, as the planner uses them at run time
        hw0 = ac.adaptcore_get_hw()
        train_keys, test_keys = split_shapes({(r["M"], r["N"], r["K"], r["dtype"]) for r in recs})
        train = [r for r in recs if (r["M"], r["N"], r["K"], r["dtype"]) in train_keys]
        test = [r for r in recs if (r["M"], r["N"], r["K"], r["dtype"]) in test_keys]
        sk = set(split_k_shapes())
        cb = set(compute_bound_shapes())
        wb = set(write_bound_shapes())
        ta = set(tall_shapes())
        from workloads import gen
        dec = {tuple(s) for s in gen.skinny_m()}
        tiny = {(r["M"], r["N"], r["K"]) for r in recs
                if max(2.0 * r["M"] * r["N"] * r["K"] / 2.5e15,
                       (2.0 * r["M"] * r["K"] + 2.0 * r["K"] * r["N"] + 2.0 * r["M"] * r["N"]) / 8e12) < 1e-6}

        def report(h):
            out = {}
            for name, rr in (("train", train), ("held_out", test)):
                out[name] = {"class": evaluate(rr, h, False), "open": evaluate(rr, h, True)}
                for tag, st in (("split_k", sk), ("compute_bound", cb), ("write_bound", wb), ("tall", ta),
                                ("decode", dec), ("floor_below_1us", tiny)):
                    sub = [r for r in rr if (r["M"], r["N"], r["K"]) in st]
                    if sub:
                        out[name][tag] = evaluate(sub, h, False)
            return out
        before = report(hw0)
        near = float(argv[argv.index("--near") + 1]) if "--near" in argv else None
        only = {config_of(r["key"]) for r in train if r["family"] == fam} if fam else None
        h, stats = fit(train, hw0, log=lambda m: print(m, file=sys.stderr), near=near, only=only)
        after = report(h)
        out = {"profile": h.as_dict(), "fit": stats, "near": near, "before": before, "after": after,
               "records": len(recs), "shapes": len(_by_shape(recs)), "train_shapes": len(train_keys),
               "held_out_shapes": len(test_keys)}
        print(json.dumps(out, indent=1))
    elif len(argv) >= 2 and argv[0] == "emit":
        with open(argv[1]) as f:
            print(emit_cpp(json.load(f)["profile"]))
    else:
        print(__doc__)


if __name__ == "__main__":
    main(sys.argv[1:])
