"""The Chrome trace-event form of a ring timeline (kvx.trace_chrome), on a
hand-made record: one complete event per interval, one named track per fill or
drain thread and per device activity, microseconds from the first start."""
import json

import paper_2609_11744_amd as kvx


def test_trace_chrome_tracks_and_times():
    ev = [
        {"kind": "fill", "piece": 0, "lane": 1, "slot": 0, "bytes": 4096, "t0_ns": 5_000,
         "t1_ns": 9_000},
        {"kind": "fill", "piece": 0, "lane": 0, "slot": 0, "bytes": 4096, "t0_ns": 6_000,
         "t1_ns": 8_000},
        {"kind": "wait", "piece": 0, "lane": 0, "slot": 0, "bytes": 0, "t0_ns": 6_500,
         "t1_ns": 9_100},
        {"kind": "h2d", "piece": 0, "lane": 0, "slot": 0, "bytes": 8192, "t0_ns": 10_000,
         "t1_ns": 12_000},
        {"kind": "scatter", "piece": 0, "lane": 0, "slot": 0, "bytes": 8192, "t0_ns": 12_500,
         "t1_ns": 13_000},
    ]
    t = kvx.trace_chrome(ev, name="restore")
    json.dumps(t)  # serialisable
    xs = [e for e in t["traceEvents"] if e["ph"] == "X"]
    assert len(xs) == len(ev)
    assert xs[0]["ts"] == 0 and xs[0]["dur"] == 4.0
    assert [x["ts"] for x in xs] == [0.0, 1.0, 1.5, 5.0, 7.5]
    names = {e["tid"]: e["args"]["name"] for e in t["traceEvents"]
             if e["ph"] == "M" and e["name"] == "thread_name"}
    assert names[xs[0]["tid"]] == "fill thread 1" and names[xs[1]["tid"]] == "fill thread 0"
    assert len({xs[3]["tid"], xs[4]["tid"], xs[2]["tid"], xs[0]["tid"]}) == 4
    assert any(e["ph"] == "M" and e["name"] == "process_name" and e["args"]["name"] == "restore"
               for e in t["traceEvents"])
    assert kvx.TRACE_KINDS[1] == "fill" and kvx.TRACE_KINDS[6] == "scatter"
