"""Host logic of the timeline metrics on a hand-built trace (no GPU)."""
import numpy as np
import pytest

from paper_2609_21483_amd import timeline as TL

DT = [("kind", "i4"), ("ticket", "i4"), ("xcd", "i4"), ("id", "i8"), ("t0", "i8"), ("t1", "i8"), ("t2", "i8")]


def rec(kind, ticket, t0, t1, t2, id_=0):
    return (kind, ticket, 0, id_, t0, t1, t2)


def us(x):
    return int(round(x * TL.TICKS_PER_US))


def test_hand_built_timeline():
    # two workgroups over 10 us; worker 0 moves, worker 1 computes
    #   worker 0: dispatch [1,3) by two waves [1,2) and [1.5,3); combine
    #   claimed at 7, copying [8,10)
    #   worker 1: a tile claimed at 1, inputs ready at 2, done at 9
    r = [rec(1, 0, us(0), us(1), us(10), 1), rec(1, 1, us(0), us(1), us(10), 0),
         rec(5, 0, us(1), us(1.8), us(2)), rec(5, 0, us(1.5), us(2.5), us(3)),
         rec(4, 0, us(7), us(8), us(10)),  # claimed at 7, waits for its row tiles until 8
         rec(2, 1, us(1), us(2), us(9))]
    m = TL.metrics(np.array(r, dtype=DT))
    assert m["layer_us"] == pytest.approx(10.0)
    assert m["prologue_us"] == pytest.approx(1.0)
    # movement [1,3) u [8,10) = 4 us; compute [2,9) = 7 us; both: [2,3) u [8,9) = 2 us
    assert m["movement_active_us"] == pytest.approx(4.0)
    assert m["compute_active_us"] == pytest.approx(7.0)
    assert m["overlap"] == pytest.approx(0.2)
    assert m["overlap_of_mov"] == pytest.approx(0.5)
    # worker 0 busy 4 us, worker 1 busy 7 us, over 2 x 10 us
    assert m["sm_active"] == pytest.approx(11.0 / 20.0)
    assert (m["workers"], m["movement_workers"]) == (2, 1)


def test_worker_busy_is_a_union_per_workgroup():
    # a worker stealing movement while its tile waits: overlapping intervals
    # of one workgroup count once
    r = [rec(1, 0, us(0), us(0.5), us(4), 0),
         rec(5, 0, us(0.5), us(1), us(2)), rec(2, 0, us(0.5), us(1.5), us(4))]
    m = TL.metrics(np.array(r, dtype=DT))
    assert m["sm_active"] == pytest.approx(3.5 / 4.0)
    assert m["overlap"] == pytest.approx(0.5 / 4.0)


def test_empty_trace():
    assert TL.metrics(np.zeros(0, dtype=DT)) is None


def test_ablation_summary_table():
    A = pytest.importorskip("paper_2609_21483_amd.ablation", reason="libmoe.so not built")
    m = {"sm_active": 0.9, "overlap": 0.05, "overlap_of_mov": 0.4, "prologue_us": 15.0}
    r = {"workload": "w", "times_us": {"serial": 100.0, "no_T": 120.0, "full": 90.0, "static": 130.0,
                                       "best_static": 110.0},
         "plans": {"no_T": (32, 1, 0, 0), "best_static": (24, 1, 0, 0)},
         "reduction": {"S": -0.2, "T": 0.25, "S+T": 0.1},
         "accuracy": {"pick": [32, 1], "t_pick_us": 90.0, "best": [24, 1], "t_best_us": 88.0, "gap": 90 / 88 - 1},
         "timeline": {"full": m, "no_T": None},
         # (c, K, n_steal, final_all, measured us, predicted us)
         "grid": [[24, 1, 3, 1, 88.0, 95.0], [24, 2, 2, 1, 93.5, 97.0], [32, 1, 4, 1, 90.0, 94.0],
                  [32, 2, 3, 1, 91.25, 96.0]]}
    md = A.markdown([r])
    assert "| w | 100.0 | 120.0 (c 32) | 90.0 | 130.0 | 110.0 (24) | -20.0% | +25.0% | +10.0% |" in md
    assert "| w | (32, 1) | 90.0 | (24, 1) | 88.0 | 2.3% |" in md
    assert "| w | full | 90.0% | 5.0% | 40.0% | 15.0 |" in md
    # the Fig 7b grid: rows c, columns K, measured (predicted), the fastest point in bold
    assert "| c | K = 1 | K = 2 |" in md
    assert "| 24 | **88.0 (95)** | 93.5 (97) |" in md
    assert "| 32 | 90.0 (94) | 91.2 (96) |" in md


def test_read_trace_decodes_wavefront_segments():
    torch = pytest.importorskip("torch")
    B = pytest.importorskip("paper_2609_21483_amd.binding", reason="libmoe.so not built")
    nseg, cap = 3, 2
    hdr = 64 + ((4 * nseg + 63) // 64) * 64
    buf = np.zeros(hdr + nseg * cap * 32, dtype=np.uint8)
    buf[:16].view(np.int32)[:] = [B.TRACE_MAGIC, nseg, cap, hdr // 8]
    buf[64:64 + 4 * nseg].view(np.int32)[:] = [1, 0, 5]  # the last count exceeds cap: cap records are kept
    recs = buf[hdr:].view(np.int64).reshape(nseg, cap, 4)

    def word0(kind, ticket, xcd, id_):
        return kind | (ticket << 8) | (xcd << 20) | (id_ << 32)

    recs[0, 0] = [word0(2, 7, 3, (1 << 24) | 5), 10, 20, 30]
    recs[1, 0] = [word0(9, 9, 9, 9), 0, 0, 0]  # beyond segment 1's count: not a record
    recs[2, 0] = [word0(5, 255, 7, 4 | (3 << 24)), 1, 2, 3]
    recs[2, 1] = [word0(1, 4095, 0, 1), 4, 5, 6]
    tr = B.read_trace(torch.from_numpy(buf))
    assert list(tr["kind"]) == [2, 5, 1]
    assert list(tr["ticket"]) == [7, 255, 4095]
    assert list(tr["xcd"]) == [3, 7, 0]
    assert list(tr["id"]) == [(1 << 24) | 5, 4 | (3 << 24), 1]
    assert list(tr["t0"]) == [10, 1, 4] and list(tr["t2"]) == [30, 3, 6]
    buf[:4] = 0  # no launch wrote the header
    assert len(B.read_trace(torch.from_numpy(buf))) == 0
