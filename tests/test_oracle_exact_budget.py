"""The oracle's information-only exact form against the layer as defined.

The layer rounds H and y to bf16 (reading R5); the exact form
(layer_with_routing_ex with round_h=False, and its unrounded y64) rounds
neither.  The distance between the two shows how much of the end-to-end
relative-L2 bar (2e-3) the two roundings take before any GPU error: on the
small parity shape and on the DBRX decode token (4 of 16 experts, d 6144).
Run with -s to see the numbers.  Measured: each rounding alone costs about
1.7e-3 and the two together about 2.4e-3 -- more than the bar -- which is
why the end-to-end bar is taken against the layer as defined (H rounded,
y unrounded: y64), and why every element is checked against a bound of its
own.  The bounds below are the roundings' own: bf16 has 8 significant bits,
so rounding y moves an element by at most 2^-8 of its value."""
import numpy as np
import pytest

import moe_inputs as mi
import oracle
from harness import bf16_f64, host_experts, rel_l2


@pytest.mark.parametrize("name", ["tiny", "decode"])
def test_rounding_share_of_the_parity_bar(name):
    wl = mi.WORKLOADS[name]
    x = wl.x()
    lg = oracle.router_logits(x, wl.router(), wl.bias())
    idx, w = oracle.route_from_logits(lg, wl.k)
    G, U, D = host_experts(wl, sorted(set(idx.ravel().tolist())))
    y_exact, _, _ = oracle.layer_with_routing_ex(x, idx, w, G, U, D, round_h=False)
    y64, y16, _ = oracle.layer_with_routing_ex(x, idx, w, G, U, D)
    y = bf16_f64(y16)
    r_h = rel_l2(y64, y_exact)       # what rounding H costs
    r_y = rel_l2(y, y64)             # what rounding y costs
    r_all = rel_l2(y, y_exact)
    print(f"{name}: rel L2 of rounding H {r_h:.3e}, of rounding y {r_y:.3e}, both {r_all:.3e} "
          f"(bar 2e-3)")
    assert np.all(np.abs(y - y64) <= np.abs(y64) * 2.0 ** -8)
    assert r_y <= 2.0 ** -8
    assert 0 < r_h < 2e-3 and 0 < r_y < 2e-3
    # the two roundings are independent: their squares add (within 20 %)
    assert abs(r_all ** 2 - (r_h ** 2 + r_y ** 2)) <= 0.2 * r_all ** 2
