"""Build windows and single-plan batches from the JSON fixtures in
tests/golden/ (named nodes, devices and models)."""
import json
import os

import numpy as np

from paper_2609_03335_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name + ".json")) as f:
        spec = json.load(f)
    devs = [d["name"] for d in spec["devices"]]
    models = [m["name"] for m in spec["models"]]
    D = len(devs)
    b = W._Builder()
    names, lat_rows, mem_rows = [], [], []
    for wf in spec["workflows"]:
        local = {n["name"]: j for j, n in enumerate(wf["nodes"])}
        b.add_workflow([[local[p] for p in n["parents"]] for n in wf["nodes"]],
                       [models.index(n["model"]) for n in wf["nodes"]])
        for n in wf["nodes"]:
            names.append(wf["name"] + "." + n["name"])
            lat_rows.append(n["lat_us"])
            mem_rows.append(n["mem_mib"])
    act_wf, act_model, off, idx, nw = b.finish()
    n = len(names)
    order = np.lexsort((np.array(b.local), np.array(b.wf_of), W._depths(n, b.parents, range(n))))
    names = [names[k] for k in order]
    index = {nm: i for i, nm in enumerate(names)}
    win = W.Window(
        n_act=n, n_wf=nw, n_models=len(models), n_dev=D, act_wf=act_wf, act_model=act_model,
        pred_off=off, pred_idx=idx,
        lat_us=np.asarray(lat_rows, np.int32)[order].reshape(-1),
        mem_mib=np.asarray(mem_rows, np.int32)[order].reshape(-1),
        wf_arrival_us=np.array([wf["arrival_us"] for wf in spec["workflows"]], np.int64),
        dev_cap_mib=np.array([d["cap_mib"] for d in spec["devices"]], np.int32),
        model_mib=np.array([m["mib"] for m in spec["models"]], np.int32),
        load_us=np.array([m["load_us"] for m in spec["models"]], np.int32).reshape(-1),
        init_resident=np.zeros(D, np.uint64), dev_free0_us=np.zeros(D, np.int64),
        w_makespan=1.0, w_p95=0.5, name=name)
    batch = [d.get("batch", 1) for d in spec["devices"]]
    if any(b != 1 for b in batch):
        win.dev_batch = np.array(batch, np.int32)
    if any("replica_cap" in m for m in spec["models"]):
        win.model_replica_cap = np.array([m.get("replica_cap", D) for m in spec["models"]], np.int32)
    if "slack_us" in spec:
        win.prefetch_slack_us = int(spec["slack_us"])
    for dname, mnames in spec.get("init_resident", {}).items():
        bits = 0
        for mn in mnames:
            bits |= 1 << models.index(mn)
        win.init_resident[devs.index(dname)] = np.uint64(bits)
    plans = {}
    for pname, ps in spec["plans"].items():
        dev = np.array([[devs.index(ps["device"][nm]) for nm in names]], np.int8)
        prio = np.array([[ps["order"].index(nm) for nm in names]], np.uint16)
        fuse = np.array([[nm in ps["fuse"] for nm in names]])
        pf = np.array([[nm in ps["prefetch"] for nm in names]])
        plans[pname] = W.PlanBatch(dev, prio, W.pack_flags(fuse, pf))
    return win, plans, index, spec
