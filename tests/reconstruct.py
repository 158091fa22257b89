"""Black-box reconstruction of a vendor GEMM's order as a descriptor (the
paper's Sec. 4 method applied to hipBLASLt on gfx950).  Test infrastructure:
it scores candidate descriptors with the CPU oracle against outputs the
vendor library computes live on the GPU, and stores no vendor output.

The procedure, per (M, N, K):
  1. candidates: the orders a tiled GEMM kernel can realise with the
     16x16x32 bf16 instruction (chunks of 8 products folded per step):
       - one carried accumulator over k in order;
       - every instruction's group rounded on its own and added to the
         accumulator (fma = 0), in groups of 32 or of 16;
       - a contiguous split-K into S parts, each part an accumulator started
         at zero, cut either by the span rule (ceil(K/S) rounded up to the
         unroll u) or balanced (the ceil(K/u) unroll steps dealt as evenly
         as they go, the first parts taking one more), merged in part order
         or by the count-up tree;
         - a strided split, k tiles of w (32 to 512) dealt round-robin over S
         wave groups;
     candidates that split k into the same parts with the same merge are
     listed once (a tree over two or three parts is the chain);
  2. the walk (Sec. 4, contiguous grouping): every column of B holds a small
     r at k = 0 and a cancelling pair +L, -L at (m, m + 1), A is all ones;
     r reaches the output exactly when the pair cancels inside a part or
     subtree that meets r's only afterwards, so the outputs over m read the
     part boundaries and the merge.  m runs over the offsets in every 64-k
     tile that sit at or straddle the chunk, group and tile boundaries the
     candidates can have.  The walk is read twice, in the first columns and
     reversed in the last ones, and on several rows: a descriptor fixes one
     order for every output, so if these differ the vendor's order depends
     on the output position (a split that changes from tile to tile) and the
     procedure stops with no survivor;
  3. fresh draws: each column holds r, +L and -L at random distinct k, which
     separates what the walk left (strided deals, group sizes), repeated
     until one candidate is left or the draws are exhausted.
Candidates whose oracle outputs differ from the vendor's in any bit are
dropped.  The result is the list of survivors (ideally one).
"""
import numpy as np

import oracle
from paper_2609_11356_amd import inputs

SPLITS = (2, 3, 4, 6, 8, 16)
UNROLLS = (64, 128, 256, 512)
STRIDED_S = (2, 4, 8)
STRIDED_W = (32, 64, 128, 256, 512)

# bf16 bit patterns: L = 2^20 and r = 2^-5, under half an fp32 ulp at L
BIG = 0x4980
NEG_BIG = 0xC980
SMALL = 0x3D00
ONE = 0x3F80
WALK_OFFSETS = (0, 7, 8, 15, 16, 31, 32, 47, 63)


def _span_cuts(K, S, u):
    span = -(-K // S)
    span = -(-span // u) * u
    cuts = [s * span for s in range(1, S)]
    return cuts if cuts and cuts[-1] < K else None


def _balanced_cuts(K, S, u):
    n = -(-K // u)
    if n < S:
        return None
    steps = [n // S + (1 if s < n % S else 0) for s in range(S)]
    cuts, at = [], 0
    for s in range(S - 1):
        at += steps[s] * u
        cuts.append(at)
    return cuts if cuts[-1] < K else None


def _parts(desc, K):
    """The parts as tuples of [begin, end) k ranges (adjacent ranges merged)."""
    S = desc.get("split_k", 1)
    if S == 1:
        return ((0, K),),
    if desc.get("split_layout") == "strided":
        w = desc["split_tile"]
        out = []
        for s in range(S):
            rs = []
            for t in range(s, -(-K // w), S):
                b, e = t * w, min((t + 1) * w, K)
                if rs and rs[-1][1] == b:
                    rs[-1] = (rs[-1][0], e)
                else:
                    rs.append((b, e))
            out.append(tuple(rs))
        return tuple(out)
    cuts = [0] + list(desc["k_cuts"]) + [K]
    return tuple(((cuts[s], cuts[s + 1]),) for s in range(S))


def _key(desc, K):
    parts = _parts(desc, K)
    merge = desc.get("split_combine", "seq") if len(parts) > 3 else "seq"
    return (desc.get("fma", 1), desc.get("mma"), parts, merge)


def candidates(K):
    """Descriptor dicts (bf16 output), one per distinct order."""
    out = [dict(mma="16x16x32", tile_k=64), dict(mma="16x16x32", tile_k=64, fma=0),
           dict(mma="32x32x16", tile_k=64, fma=0)]
    for S in SPLITS:
        for u in UNROLLS:
            for cuts in (_span_cuts(K, S, u), _balanced_cuts(K, S, u)):
                if cuts is None:
                    continue
                for sc in ("seq", "tree"):
                    out.append(dict(mma="16x16x32", tile_k=64, split_k=S, k_cuts=cuts, split_combine=sc))
    for S in STRIDED_S:
        for w in STRIDED_W:
            if -(-K // w) < S:
                continue                  # some wave group would get no tile
            for sc in ("seq", "tree"):
                out.append(dict(mma="16x16x32", tile_k=min(w, 64), split_k=S, split_layout="strided",
                                split_tile=w, split_combine=sc))
    seen, uniq = set(), []
    for d in out:
        k = _key(d, K)
        if k not in seen:
            seen.add(k)
            d["out"] = "bf16"
            uniq.append(d)
    return uniq


def vendor_gemm(A, B):
    """C = A . B by torch.matmul (hipBLASLt on ROCm), bf16 bits."""
    import torch
    to = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()
    C = torch.matmul(to(A), to(B))
    torch.cuda.synchronize()
    return C.view(torch.int16).cpu().numpy().view(np.uint16)


def walk_positions(K):
    """Pair positions m of the walk (the pair sits at m and m + 1)."""
    m = {64 * t + o for t in range(-(-K // 64)) for o in WALK_OFFSETS}
    return np.array(sorted(x for x in m if 1 <= x <= K - 2), dtype=np.int64)


def walk_columns(K, ms):
    B = np.zeros((K, len(ms)), dtype=np.uint16)
    c = np.arange(len(ms))
    B[0, c] = SMALL
    B[ms, c] = BIG
    B[ms + 1, c] = NEG_BIG
    return B


def triple_columns(K, n, rng):
    B = np.zeros((K, n), dtype=np.uint16)
    for c in range(n):
        p, q, s = rng.choice(K, 3, replace=False)
        B[p, c], B[q, c], B[s, c] = SMALL, BIG, NEG_BIG
    return B


def _same(want, got):
    nan = ((want & 0x7FFF) > 0x7F80) & ((got & 0x7FFF) > 0x7F80)
    return (want == got) | nan


def vendor_probe(M, N, K, Bcols, vendor, reverse=False):
    """The vendor's outputs for the probe columns Bcols (K x n) run at the
    (M, N, K) shape, in batches of N columns with A all ones; the probes go
    to the first columns of each batch, or to the last in reverse order.
    Returns (outputs of row 0 per probe, whether every row agreed)."""
    A = np.full((M, K), ONE, dtype=np.uint16)
    rows = sorted({0, M // 2, M - 1})
    n = Bcols.shape[1]
    got = np.zeros(n, dtype=np.uint16)
    rows_agree = True
    for b in range(0, n, N):
        blk = Bcols[:, b:b + N]
        w = blk.shape[1]
        cols = N - 1 - np.arange(w) if reverse else np.arange(w)
        B = np.zeros((K, N), dtype=np.uint16)
        B[:, cols] = blk
        C = vendor(A, B)
        for i in rows:
            rows_agree &= bool(_same(C[i, cols], C[0, cols]).all())
        got[b:b + w] = C[0, cols]
    return got, rows_agree


def oracle_probe(desc, Bcols):
    """The candidate's outputs for the probe columns (one row of ones)."""
    K, n = Bcols.shape
    A = np.full((1, K), ONE, dtype=np.uint16)
    jj = np.arange(n, dtype=np.int64)
    return inputs.f32_to_bf16_bits(oracle.gemm_at(desc, A, Bcols, None, np.zeros_like(jj), jj, M=1))


def reconstruct(M, N, K, draws=3, triples=512, seed=0, log=print, vendor=None):
    """Run the procedure; returns (survivors, history, uniform).  history
    lists the number of candidates before the walk, after it and after each
    draw.  uniform is False when the vendor's order depends on the output
    position (the walk read at the first columns and, reversed, at the last
    ones differ, or rows with equal A differ): no single descriptor can then
    hold and the survivors are empty.  vendor(A, B) -> bf16 bits of A . B;
    torch.matmul unless given."""
    vendor = vendor or vendor_gemm
    pool = candidates(K)
    history = [len(pool)]
    ms = walk_positions(K)
    walk = walk_columns(K, ms)
    got, rows_agree = vendor_probe(M, N, K, walk, vendor)
    got_rev, rows_agree_rev = vendor_probe(M, N, K, walk, vendor, reverse=True)
    uniform = rows_agree and rows_agree_rev and bool(_same(got, got_rev).all())
    if not uniform:
        log("  the vendor's order depends on the output position")
        return [], history, False
    pool = [d for d in pool if _same(oracle_probe(d, walk), got).all()]
    history.append(len(pool))
    log("  walk over %d pair positions: %d candidates left" % (len(ms), len(pool)))
    rng = np.random.default_rng(seed)
    for d in range(draws):
        if len(pool) <= 1:
            break
        probes = triple_columns(K, triples, rng)
        got, _ = vendor_probe(M, N, K, probes, vendor)
        pool = [c for c in pool if _same(oracle_probe(c, probes), got).all()]
        history.append(len(pool))
        log("  draw %d: %d candidates left" % (d, len(pool)))
    return pool, history, True


def describe(desc):
    S = desc.get("split_k", 1)
    if S == 1:
        if desc.get("fma", 1):
            return "one carried accumulator"
        return "groups of %d rounded alone (fma = 0)" % (32 if desc["mma"] == "16x16x32" else 16)
    if desc.get("split_layout") == "strided":
        return "strided split S = %d, w = %d, %s merge" % (S, desc["split_tile"], desc["split_combine"])
    return "contiguous split S = %d at %s, %s merge" % (S, list(desc["k_cuts"]), desc["split_combine"])


# ---------------------------------------------------------------- the table
# Widths from the paper's model table (App. C): (N, K) of the MLP, MoE and
# projection GEMMs (up: N = FFN or expert width, K = hidden; down: the
# reverse), run at token counts M.
APPC_PAIRS = [(2880, 2880), (1856, 2688), (2688, 1856), (6144, 2048), (2048, 6144), (2048, 768), (3072, 7168),
              (7168, 3072), (5120, 17408), (17408, 5120), (12800, 4096), (10240, 2048), (7168, 18432),
              (512, 2048), (2048, 512), (1536, 3072), (4096, 4096), (4096, 14336)]
APPC_TOKENS = [1, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048]


def sweep(out_path, pairs=APPC_PAIRS, tokens=APPC_TOKENS):
    """Reconstruct every shape; writes JSON with, per shape, the survivors
    and the number of vendor calls made (in call order, so that a kernel
    trace of the same run can be joined call by call)."""
    import json
    calls = []

    def counted(shape):
        def f(A, B):
            calls.append(shape)
            return vendor_gemm(A, B)
        return f

    res = []
    for N, K in pairs:
        for M in tokens:
            pool, hist, uniform = reconstruct(M, N, K, draws=4, seed=M + N + K, log=lambda s: None,
                                              vendor=counted([M, N, K]))
            res.append(dict(M=M, N=N, K=K, history=hist, uniform=uniform,
                            survivors=[describe(d) for d in pool]))
            print("%5d x %5d x %5d  %-60s %s" % (M, N, K, res[-1]["survivors"] if uniform else "order varies by output",
                                                 hist), flush=True)
    with open(out_path, "w") as f:
        json.dump(dict(shapes=res, calls=calls), f)


def _name_field(name, key):
    import re
    m = re.search(r"_" + key + r"([0-9x_n]+?)(?=_[A-Z]|$)", name)
    return m.group(1) if m else "?"


def join(orders_path, trace_csv):
    """Markdown table: shape, the vendor kernel's macro tile (MT), workgroup
    shape (WG, whose last factor is the local split of k) and the
    reconstructed order; the i-th GEMM kernel of the trace is the i-th
    vendor call of the sweep."""
    import csv
    import json
    d = json.load(open(orders_path))
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    gemm = [r for r in rows if r["Kernel_Name"].startswith("Cijk")]
    if len(gemm) != len(d["calls"]):
        raise SystemExit("%d GEMM kernels in the trace, %d vendor calls" % (len(gemm), len(d["calls"])))
    kern = {}
    for r, c in zip(gemm, d["calls"]):
        n = r["Kernel_Name"]
        wgs = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]) * int(r["Workgroup_Size_Y"]) *
                                             int(r["Workgroup_Size_Z"]))
        k = (_name_field(n, "MT"), _name_field(n, "WG"), wgs)
        kern.setdefault(tuple(c), set()).add(k)
    print("| M | N | K | MT | WG | workgroups | tiles | order |")
    print("|---|---|---|---|---|---|---|---|")
    for s in d["shapes"]:
        ks = kern[(s["M"], s["N"], s["K"])]
        (mt, wg, wgs), = ks if len(ks) == 1 else [("several", "", 0)]
        try:
            t0, t1 = (int(x) for x in mt.split("x")[:2])
            tiles = -(-s["N"] // t0) * -(-s["M"] // t1)
        except ValueError:
            tiles = "?"
        order = "; ".join(s["survivors"]) if s["uniform"] else "varies by output tile"
        if s["uniform"] and len(s["survivors"]) != 1:
            order = "%d survivors: %s" % (len(s["survivors"]), order)
        print("| %d | %d | %d | %s | %s | %d | %s | %s |" % (s["M"], s["N"], s["K"], mt, wg, wgs, tiles, order))


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--out", help="run the sweep on the GPU and write its JSON here")
    ap.add_argument("--join", nargs=2, metavar=("ORDERS_JSON", "KERNEL_TRACE_CSV"),
                    help="print the table of a sweep joined with a kernel trace of the same run")
    a = ap.parse_args()
    if a.out:
        sweep(a.out)
    if a.join:
        join(*a.join)
