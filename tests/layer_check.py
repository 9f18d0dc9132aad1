"""Sampled comparison of one convolution layer's outputs with the oracle at
full workload sizes (test infrastructure)."""
import oracle
from helpers import TOL_F32, assert_close


def _geom(L):
    return dict(stride=L.s, pad=L.p, group=L.g)


def check_layer_sampled(L, x, w, b, top, top_diff, dx, dw, db, images, filters, tol=TOL_F32,
                        what="", dx_mask=None, db_top_diff=None):
    """x, w, b, top_diff: the operands the GPU layer consumed (numpy);
    top, dx, dw, db: its outputs.  dx may be None (not computed).  dx_mask:
    the data gradient was stored times this mask (a fused ReLU backward).
    db_top_diff: the top gradient the bias gradient sums, when it differs
    from the one the products used (bf16 operands round the latter)."""
    print(f"check {what}: images {images} filters {filters}", flush=True)
    xs = x[images]
    y_ref = oracle.conv_forward(xs, w, b, L.s, L.p, L.g, L.relu)
    assert_close(top[images], y_ref, tol, f"{what} forward")
    if top_diff is None:
        return
    topm = top if L.relu else None
    if dx is not None:
        dx_ref, _, _ = oracle.conv_backward(xs, w, top_diff[images],
                                            top=None if topm is None else topm[images],
                                            relu=L.relu, need=("dx",), **_geom(L))
        if dx_mask is not None:
            dx_ref = dx_ref * dx_mask[images]
        assert_close(dx[images], dx_ref, tol, f"{what} data gradient")
    # bias gradient of every filter (the oracle's db loop alone is cheap at full size)
    gdb = top_diff if db_top_diff is None else db_top_diff
    _, _, db_ref = oracle.conv_backward(x, w, gdb, top=topm, relu=L.relu, need=("db",),
                                        **_geom(L))
    assert_close(db, db_ref, tol, f"{what} bias gradient")
    Kg, Cg = L.K // L.g, L.C // L.g
    for k in filters:
        t = k // Kg
        _, dw_ref, _ = oracle.conv_backward(
            x[:, t * Cg:(t + 1) * Cg], w[k:k + 1], top_diff[:, k:k + 1],
            top=None if topm is None else topm[:, k:k + 1], relu=L.relu, stride=L.s, pad=L.p,
            need=("dw",))
        assert_close(dw[k:k + 1], dw_ref, tol, f"{what} weight gradient filter {k}")
