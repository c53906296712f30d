"""The stepped MFMA kernel's launch-shape rule for register tables, stated independently of
the library's host code so that tests can check the library against it."""


def stepped_shape(m, k, n):
    """The launch shape the library gives the stepped kernel with register tables (fitted
    codebooks): (64-row workgroups, batch tiles per workgroup column, K parts). Every shape whose
    grid has at most 256 workgroups competes on (steps per workgroup) x (per-step time), per-step
    time 0.5 + 0.3 t us for 128 rows and 0.376 + 0.184 t us for 64 rows, plus 5 us for two K
    parts (allowed from 16 steps of 256); with none that fits, 128-row workgroups with
    min(ceil(m / 16), 8) tiles."""
    t0 = min(-(-m // 16), 8)
    gy = -(-m // 128) if m > 128 else 1
    best, best_cost = ((-(-n // 64)) * gy <= 256, t0, 1), None
    steps = -(-k // 256)
    for rows in (128, 64):
        t = t0
        while True:
            for parts in ((1, 2) if steps >= 16 else (1,)):
                if -(-n // rows) * -(-m // (16 * t)) * parts > 256:
                    continue
                per = 0.5 + 0.3 * t if rows == 128 else 0.376 + 0.184 * t
                cost = -(-steps // parts) * per + (5.0 if parts == 2 else 0.0)
                if best_cost is None or cost < best_cost:
                    best, best_cost = (rows == 64, t, parts), cost
            if t == 1:
                break
            t = (t + 1) // 2
    return best


def stepped_name(m, k, n):
    narrow, t, _ = stepped_shape(m, k, n)
    coal = "true" if t <= 2 else "false"
    if narrow:
        return f"k_mfma2_narrow<4, {t}, false, {coal}>"
    return f"k_mfma2<4, {t}, 4, false, {coal}>"
