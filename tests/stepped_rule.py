"""The stepped MFMA kernel's launch-shape rule, stated independently of the library's host code
so that tests can check the library against it."""

# Per-step time of a workgroup (us per step of 256 k) with t batch tiles: fixed + tile * t, for
# 64- and 128-row workgroups, and the extra cost of two K parts (us), per kind of
# dequantization: register tables (fitted 4-bit codebooks), the 4-bit LDS table (any other
# 4-bit codebook) and 8-bit codes.
COSTS = {
    "register": (0.376, 0.184, 0.500, 0.300, 5.0),
    "table4": (0.283, 0.198, 0.205, 0.374, 3.1),
    "bits8": (0.422, 0.279, 0.156, 0.600, 3.0),
}


def stepped_shape(m, k, n, kind="register"):
    """(64-row workgroups, batch tiles per workgroup column, K parts). Every shape whose grid
    has at most 256 workgroups competes on (steps per workgroup) x (per-step time), plus the
    cost of two K parts (allowed from 16 steps of 256); t runs t0, ceil(t0 / 2), ... 1 with
    t0 = min(ceil(m / 16), cap), cap 8 for register tables and 4 otherwise; 8-bit codes never
    take 128-row workgroups with one tile. With no shape that fits: 128-row workgroups with t0
    tiles, unless 64-row ones fit."""
    f64, t64, f128, t128, two = COSTS[kind]
    cap = 8 if kind == "register" else 4
    t0 = min(-(-m // 16), cap)
    gy = -(-m // (16 * cap)) if m > 16 * cap else 1
    best, best_cost = ((-(-n // 64)) * gy <= 256, t0, 1), None
    steps = -(-k // 256)
    for rows in (128, 64):
        t = t0
        while True:
            for parts in ((1, 2) if steps >= 16 else (1,)):
                if kind == "bits8" and rows == 128 and t == 1:
                    continue     # left out for 8-bit codes
                if -(-n // rows) * -(-m // (16 * t)) * parts > 256:
                    continue
                per = f128 + t128 * t if rows == 128 else f64 + t64 * t
                cost = -(-steps // parts) * per + (two if parts == 2 else 0.0)
                if best_cost is None or cost < best_cost:
                    best, best_cost = (rows == 64, t, parts), cost
            if t == 1:
                break
            t = (t + 1) // 2
    return best


def stepped_name(m, k, n, kind="register"):
    narrow, t, _ = stepped_shape(m, k, n, kind)
    bits = 8 if kind == "bits8" else 4
    pairs = "false" if kind == "register" else "true"
    coal = "true" if t <= 2 else "false"
    if narrow:
        return f"k_mfma2_narrow<{bits}, {t}, {pairs}, {coal}>"
    return f"k_mfma2<{bits}, {t}, 4, {pairs}, {coal}>"
