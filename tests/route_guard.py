"""Guard bands of end-to-end routing: when two predictions of the same stages agree only to the
predictor tolerance, their routes may legitimately differ. A prediction enters routing in two
places: the demand R_kv tested against each node's headroom, and the decode term of the latency
score (Eq. 2), which is the same for every node of a stage and so reorders nodes only through
float32 rounding. Every difference between two routes must be one of those."""
import numpy as np


def explain_route_differences(w, rows, pred_a, kv_a, idx_a, kv_b, idx_b):
    """Route lists idx_a (from prediction a) and idx_b (from prediction b) of the stages ``rows``
    of workload ``w``. Asserts that every stage whose lists differ has a node whose feasibility
    flips between the two demands, or, at the first differing position, two nodes whose scores
    under prediction a are within two float32 ulps. Returns (fraction identical, flips, ties)."""
    same = np.all(idx_a == idx_b, axis=1)
    rho = w.spec.rho
    need_a = kv_a if rho == 0 else kv_a * (1 + rho)
    need_b = kv_b if rho == 0 else kv_b * (1 + rho)
    model = w.model_id[rows]
    ks = (pred_a * w.decode_s_per_token[model]).astype(np.float32)
    resident = (w.resident_mask[None, :] >> model.astype(np.uint64)[:, None]) & np.uint64(1)
    flips = ties = 0
    for i in np.nonzero(~same)[0]:
        if np.any((need_a[i] <= w.free_bytes) != (need_b[i] <= w.free_bytes)):
            flips += 1
            continue
        j = int(np.argmax(idx_a[i] != idx_b[i]))
        a, c = int(idx_a[i, j]), int(idx_b[i, j])
        assert a >= 0 and c >= 0, f"stage {rows[i]}: the lists differ in length without a feasibility flip"

        def score(nd):
            cold = np.float32(0.0) if resident[i, nd] else w.cold_s[nd]
            return np.float32(np.float32(w.queue_s[nd] + cold) + ks[i])

        sa, sc = score(a), score(c)
        ulp = float(np.spacing(np.float32(max(abs(sa), abs(sc)))))
        assert abs(float(sc) - float(sa)) <= 2 * ulp, (
            f"stage {rows[i]}: nodes {a} / {c} with scores {sa} / {sc} under prediction a are not a rounding tie")
        ties += 1
    return float(same.mean()), flips, ties
