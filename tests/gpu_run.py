"""Run the HIP path (through the C ABI) on a synth.Workload and bring the
results back as numpy arrays shaped like the oracle's."""
from __future__ import annotations

import numpy as np
import torch

import paper_2602_16100_amd as pc


def dev(a):
    return pc.to_device(a, "cuda")


def selectors(labels, pred_off, preds, n_preds=None):
    f, p = pc.pc_eval_selectors(dev(labels), dev(pred_off), dev(preds), n_preds=n_preds)
    torch.cuda.synchronize()
    return f.cpu().numpy().view(np.uint64), p.cpu().numpy().view(np.uint32)


def affinity(labels, row_off, term_off, preds, n_terms=None, n_preds=None):
    """Feasible bitset, popcount, inventory flags and the data-error word."""
    ctx = pc.context()
    ctx.data_errors(clear=True)
    f, p, u = pc.pc_eval_affinity(dev(labels), dev(row_off), dev(term_off), dev(preds), n_terms=n_terms,
                                  n_preds=n_preds)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    return f.cpu().numpy().view(np.uint64), p.cpu().numpy().view(np.uint32), u.cpu().numpy(), flags


def preferred(labels, row_off, term_off, weight, preds, feasible=None, n_terms=None, n_preds=None):
    """Best node, score, tie count and the data-error word."""
    ctx = pc.context()
    ctx.data_errors(clear=True)
    f = None if feasible is None else torch.from_numpy(np.ascontiguousarray(feasible).view(np.int64)).cuda()
    b, s, c = pc.pc_score_preferred(dev(labels), dev(row_off), dev(term_off),
                                    dev(np.ascontiguousarray(weight, np.uint32)), dev(preds), feasible=f,
                                    n_terms=n_terms, n_preds=n_preds)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    return (b.cpu().numpy(), s.cpu().numpy().view(np.uint32), c.cpu().numpy().view(np.uint32), flags)


def _rows2d(a, Q):
    a = np.ascontiguousarray(a, np.int32)
    return a.reshape(Q, a.shape[1] if a.ndim == 2 else 1)


def synthesize(V, port_off, port_peer, region, src, target, allowed, via, forbid, key, out_port, prio, max_hops,
               weight=None, n_ports=None):
    """Hop counts, walks, rules (numpy records) and the data-error word."""
    ctx = pc.context()
    ctx.data_errors(clear=True)
    Q = src.shape[0]
    h, p, r = pc.pc_synthesize_paths(V, dev(port_off), dev(port_peer), dev(region), dev(src), dev(target),
                                     dev(allowed), dev(_rows2d(via, Q)), dev(_rows2d(forbid, Q)),
                                     dev(np.ascontiguousarray(key, np.uint32)), dev(out_port), prio, max_hops,
                                     weight=None if weight is None else dev(np.ascontiguousarray(weight, np.uint32)),
                                     n_ports=n_ports)
    torch.cuda.synchronize()
    flags = ctx.data_errors(clear=True)
    rules = r.cpu().numpy().reshape(-1).view(pc.RULE_DT).reshape(Q, -1) if Q else np.zeros((0, max_hops + 1),
                                                                                               pc.RULE_DT)
    return h.cpu().numpy(), p.cpu().numpy(), rules, flags


def trace(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, n_ports=None, n_rules=None):
    out = pc.pc_trace_flows(S, dev(port_off), dev(port_peer), dev(jur), dev(rule_off), dev(rules),
                            dev(np.ascontiguousarray(hdr, np.uint32)), dev(ingress), ttl,
                            n_ports=n_ports, n_rules=n_rules)
    torch.cuda.synchronize()
    return pc.records(out, pc.TRACE_OUT_DT)


def reach(V, adj_off, adj, region, src, allowed, target=None, n_adj=None):
    d = pc.pc_masked_reach(V, dev(adj_off), dev(adj), dev(region), dev(src), dev(allowed),
                           None if target is None else dev(target), n_adj=n_adj)
    torch.cuda.synchronize()
    return d.cpu().numpy()


def report(intents, feasible, popcnt, N, traces, expect, reach_d):
    f = torch.from_numpy(np.ascontiguousarray(feasible).view(np.int64)).cuda()
    p = torch.from_numpy(np.ascontiguousarray(popcnt).view(np.int32)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(traces).view(np.uint8).reshape(-1, 12)).cuda()
    r = torch.from_numpy(np.ascontiguousarray(reach_d, np.int32)).cuda()
    pss, reason, summ = pc.pc_report(dev(intents), f, p, N, t, dev(expect), r)
    torch.cuda.synchronize()
    return (pss.cpu().numpy().view(np.uint64), reason.cpu().numpy(),
            pc.records(summ, pc.SUMMARY_DT)[0])


def run_workload(wl):
    """All stages on the GPU, device-resident between stages (as a caller
    would chain them); outputs copied back at the end."""
    out = {}
    ctx = pc.context()
    ctx.data_errors(clear=True)
    if "labels" in wl.arrays:
        f, p = pc.pc_eval_selectors(dev(wl["labels"]), dev(wl["pred_off"]), dev(wl["preds"]))
        out["_f"], out["_p"] = f, p
    if "rules" in wl.arrays:
        out["_t"] = pc.pc_trace_flows(wl["S"], dev(wl["port_off"]), dev(wl["port_peer"]), dev(wl["jur"]),
                                      dev(wl["rule_off"]), dev(wl["rules"]), dev(wl["hdr"]), dev(wl["ingress"]),
                                      wl["ttl"])
    if "src" in wl.arrays:
        tgt = wl.arrays.get("target")
        out["_r"] = pc.pc_masked_reach(wl["V"], dev(wl["adj_off"]), dev(wl["adj"]), dev(wl["region"]),
                                       dev(wl["src"]), dev(wl["allowed"]), None if tgt is None else dev(tgt))
    if "intents" in wl.arrays:
        pss, reason, summ = pc.pc_report(dev(wl["intents"]), out["_f"], out["_p"], wl["N"], out["_t"],
                                         dev(wl["expect"]), out["_r"])
        out["pass"] = pss.cpu().numpy().view(np.uint64)
        out["reason"] = reason.cpu().numpy()
        out["summary"] = pc.records(summ, pc.SUMMARY_DT)[0]
    torch.cuda.synchronize()
    if "_f" in out:
        out["feasible"] = out.pop("_f").cpu().numpy().view(np.uint64)
        out["popcnt"] = out.pop("_p").cpu().numpy().view(np.uint32)
    if "_t" in out:
        out["traces"] = pc.records(out.pop("_t"), pc.TRACE_OUT_DT)
    if "_r" in out:
        out["reach"] = out.pop("_r").cpu().numpy()
    out["flags"] = ctx.data_errors(clear=True)
    return out


def trace_watch(S, port_off, port_peer, jur, rule_off, rules, hdr, ingress, ttl, watch):
    out, visit = pc.pc_trace_flows_watch(S, dev(port_off), dev(port_peer), dev(jur), dev(rule_off), dev(rules),
                                         dev(np.ascontiguousarray(hdr, np.uint32)), dev(ingress), ttl,
                                         dev(np.ascontiguousarray(watch, np.int32)))
    torch.cuda.synchronize()
    return pc.records(out, pc.TRACE_OUT_DT), visit.cpu().numpy().view(np.uint32)


def reach_via(V, adj_off, adj, region, src, allowed, target, via, forbid):
    d = pc.pc_masked_reach_via(V, dev(adj_off), dev(adj), dev(region), dev(src), dev(allowed), dev(target),
                               dev(np.ascontiguousarray(via, np.int32)), dev(np.ascontiguousarray(forbid, np.int32)))
    torch.cuda.synchronize()
    return d.cpu().numpy()


def report_paths(intents, feasible, popcnt, N, traces, expect, reach_d, visit, pexp):
    f = torch.from_numpy(np.ascontiguousarray(feasible).view(np.int64)).cuda()
    p = torch.from_numpy(np.ascontiguousarray(popcnt).view(np.int32)).cuda()
    t = torch.from_numpy(np.ascontiguousarray(traces).view(np.uint8).reshape(-1, 12)).cuda()
    r = torch.from_numpy(np.ascontiguousarray(reach_d, np.int32)).cuda()
    v = torch.from_numpy(np.ascontiguousarray(visit, np.uint32).view(np.int32)).cuda()
    pss, reason, summ = pc.pc_report_paths(dev(intents), f, p, N, t, dev(expect), r, v, dev(pexp))
    torch.cuda.synchronize()
    return (pss.cpu().numpy().view(np.uint64), reason.cpu().numpy(),
            pc.records(summ, pc.SUMMARY_DT)[0])


def run_paths_workload(wl):
    """All stages with the path constraints (watch lists, waypoints,
    forbidden switches), device-resident between stages."""
    out = {}
    ctx = pc.context()
    ctx.data_errors(clear=True)
    f, p = pc.pc_eval_selectors(dev(wl["labels"]), dev(wl["pred_off"]), dev(wl["preds"]))
    t, v = pc.pc_trace_flows_watch(wl["S"], dev(wl["port_off"]), dev(wl["port_peer"]), dev(wl["jur"]),
                                   dev(wl["rule_off"]), dev(wl["rules"]), dev(wl["hdr"]), dev(wl["ingress"]),
                                   wl["ttl"], dev(wl["watch"]))
    r = pc.pc_masked_reach_via(wl["V"], dev(wl["adj_off"]), dev(wl["adj"]), dev(wl["region"]), dev(wl["src"]),
                               dev(wl["allowed"]), dev(wl["target"]), dev(wl["via"]), dev(wl["forbid"]))
    pss, reason, summ = pc.pc_report_paths(dev(wl["intents"]), f, p, wl["N"], t, dev(wl["expect"]), r, v,
                                           dev(wl["pexp"]))
    torch.cuda.synchronize()
    out["feasible"] = f.cpu().numpy().view(np.uint64)
    out["popcnt"] = p.cpu().numpy().view(np.uint32)
    out["traces"] = pc.records(t, pc.TRACE_OUT_DT)
    out["visit"] = v.cpu().numpy().view(np.uint32)
    out["reach"] = r.cpu().numpy()
    out["pass"] = pss.cpu().numpy().view(np.uint64)
    out["reason"] = reason.cpu().numpy()
    out["summary"] = pc.records(summ, pc.SUMMARY_DT)[0]
    out["flags"] = ctx.data_errors(clear=True)
    return out
