"""Small builders shared by the tests (fixtures from the paper, tiny graphs)."""
from __future__ import annotations

import json
import os

import numpy as np

import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
OPS = {"In": synth.OP_IN, "NotIn": synth.OP_NOTIN, "Exists": synth.OP_EXISTS}


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def encode_label_matrix(fx):
    """Paper label matrix -> (labels uint8 [N, L], per-key value dictionary).
    Keys no node carries become all-absent columns."""
    keys = fx["keys"]
    vocab = {k: {} for k in keys}
    for node in fx["nodes"]:
        for k in keys:
            if k in node:
                vocab[k].setdefault(node[k], len(vocab[k]))
    N, L = len(fx["nodes"]), len(keys)
    labels = np.full((N, L), synth.ABSENT, np.uint8)
    for n, node in enumerate(fx["nodes"]):
        for l, k in enumerate(keys):
            if k in node:
                labels[n, l] = vocab[k][node[k]]
    return labels, vocab


def encode_selector(fx, vocab, selector):
    """[[key, op, [values]], ...] -> pc_pred records.  A value no node carries
    gets a fresh code beyond the key's vocabulary (it matches nothing)."""
    keys = fx["keys"]
    preds = np.zeros(len(selector), synth.PRED_DT)
    for j, (k, op, values) in enumerate(selector):
        preds[j]["label"] = keys.index(k)
        preds[j]["op"] = OPS[op]
        bm = [0, 0, 0, 0]
        for v in values:
            code = vocab[k].get(v)
            if code is None:
                code = len(vocab[k]) + 100
            bm[code >> 6] |= 1 << (code & 63)
        preds[j]["vals"] = np.array(bm, np.uint64)
    return preds


def bits_to_set(words, N):
    out = set()
    for n in range(N):
        if (int(words[n >> 6]) >> (n & 63)) & 1:
            out.add(n)
    return out


def line_topology(n_switch, jur, hosts_per_switch=1):
    """Switches 0..n-1 on a line; link ports (neighbour-id order) then host ports."""
    nbr = [[v for v in (s - 1, s + 1) if 0 <= v < n_switch] for s in range(n_switch)]
    return ports_topology(nbr, jur, hosts_per_switch)


def ports_topology(nbr, jur, hosts_per_switch=1):
    S = len(nbr)
    nports = np.array([len(nbr[s]) + hosts_per_switch for s in range(S)], np.int32)
    port_off = np.zeros(S + 1, np.int32)
    port_off[1:] = np.cumsum(nports)
    peer = np.full(int(port_off[-1]), -1, np.int32)
    for s in range(S):
        for i, v in enumerate(sorted(nbr[s])):
            peer[port_off[s] + i] = v
    adj_off = np.zeros(S + 1, np.int32)
    adj = []
    for s in range(S):
        adj.extend(sorted(nbr[s]))
        adj_off[s + 1] = len(adj)
    return dict(S=S, port_off=port_off, port_peer=peer, jur=np.asarray(jur, np.uint8),
                adj_off=adj_off, adj=np.asarray(adj, np.int32), nbr=[sorted(x) for x in nbr])


def exact_rule(key, action, priority=100):
    r = np.zeros(1, synth.RULE_DT)[0]
    r["value"] = key
    r["mask"] = np.array([0xFFFFFFFF] * 3 + [0xFF], np.uint32)
    r["priority"] = priority
    r["action"] = action
    return r


def tables_from_lists(per_switch):
    """list of lists of rule records -> (rule_off, rules)."""
    S = len(per_switch)
    rule_off = np.zeros(S + 1, np.int32)
    allr = []
    for s, lst in enumerate(per_switch):
        allr.extend(lst)
        rule_off[s + 1] = len(allr)
    rules = np.zeros(len(allr), synth.RULE_DT)
    for i, r in enumerate(allr):
        rules[i] = r
    return rule_off, rules


def leak_fixture():
    """The paper's transit-switch case (golden paper_transit_leak.json): three
    switches on a line, exact-match rules along the flow's path.
    Returns (fixture, topology, path, key, rule_off, rules)."""
    fx = load_golden("paper_transit_leak.json")
    names = [s["name"] for s in fx["switches"]]
    nbr = [[names.index(x) for x in s["links"]] for s in fx["switches"]]
    jur = [fx["regions"].index(s["region"]) for s in fx["switches"]]
    topo = ports_topology(nbr, jur, hosts_per_switch=1)
    path = [names.index(x) for x in fx["flow"]["path"]]
    key = np.array([0x0A000001, 0x0A000003, (4000 << 16) | 443, 6], np.uint32)
    per = [[] for _ in names]
    for i, s in enumerate(path):
        a = topo["nbr"][s].index(path[i + 1]) if i + 1 < len(path) else len(topo["nbr"][s])
        per[s].append(exact_rule(key, a))
    rule_off, rules = tables_from_lists(per)
    return fx, topo, path, key, rule_off, rules
