/*
 * pc.h -- C ABI of the GPU compliance checker (libpc.so, MI355X / gfx950).
 *
 * The library evaluates the validator checks of an LLM-driven, intent-based
 * privacy orchestration system (arXiv 2602.16100) over a post-deployment
 * state snapshot:
 *   - pc_eval_selectors : placement constraints -- node selectors over node
 *                         labels (Formal Model and Satisfaction, condition
 *                         (i) and the example intent; Kubernetes node
 *                         selector / affinity in Intent-driven
 *                         Orchestration Plane).
 *   - pc_trace_flows    : routing constraints on the paths realised by the
 *                         installed flow rules (condition (ii); per-hop flow
 *                         rules in "Network orchestration").
 *   - pc_masked_reach   : existence and hop distance of a path that stays
 *                         inside the allowed jurisdictions (the path
 *                         scheduler's graph search with BFS fallback).
 *   - pc_report         : per-intent pass/fail -- an intent passes only if
 *                         all of its checks pass (Automated Validation
 *                         Pipeline, validator check definition); an
 *                         unenforceable intent fails closed.
 *   - pc_trace_flows_watch, pc_masked_reach_via, pc_report_paths : the same
 *                         checks with required waypoints and forbidden
 *                         switches (the routing constraints of a
 *                         Configuration; must_go / forbidden lists).
 *   - pc_eval_affinity  : placement with full node affinity (OR-ed terms,
 *                         six operators, label-inventory flags).
 *   - pc_score_preferred : the best feasible node under weighted preferred
 *                         terms (secondary placement objectives).
 *   - pc_trace_flows_delta : re-traces only the traces whose walk visited a
 *                         switch whose rules changed.
 *   - pc_synthesize_paths : the step before validation -- the path
 *                         scheduler's search for a compliant path and its
 *                         compilation into per-hop flow rules.
 *
 * Conventions shared by every entry point
 *   - Every array argument is a DEVICE pointer owned by the caller; it must
 *     stay valid until the work queued on `stream` has completed.  The
 *     library keeps no pointer past the call and never frees caller memory.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every
 *     entry point is asynchronous and stream-ordered, except
 *     pc_trace_flows(_watch), which reads back the size of its rule index once and
 *     one live-trace count per hop level, and pc_data_errors and
 *     pc_profile_read, which wait for the stream.
 *   - Return value: PC_OK, or a negative PC_E* code.  Argument errors are
 *     detected on the host before any device work is queued; the message
 *     is available from pc_last_error.  No C++ exception crosses the ABI.
 *   - Malformed device data (see PC_DERR_*) never causes an out-of-bounds
 *     access: the item is given the documented neutral meaning and a bit
 *     is OR-ed into the context's sticky data-error word, read with
 *     pc_data_errors.  A flag depends only on the input arrays, not on the
 *     order of the traversal.
 *   - One context per host thread / stream; calls on one context must not
 *     overlap.  Scratch memory is owned by the context, grown on demand
 *     (growing synchronises the device) and freed by pc_destroy.
 */
#ifndef PC_H
#define PC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PC_VERSION 10

enum { PC_OK = 0, PC_EINVAL = -1, PC_ENOMEM = -2, PC_EDEVICE = -3 };

/* selector operators (Kubernetes node-affinity semantics) */
enum { PC_OP_IN = 0, PC_OP_NOTIN = 1, PC_OP_EXISTS = 2 };
/* further operators, accepted by pc_eval_affinity only */
enum { PC_OP_DOESNOTEXIST = 3, PC_OP_GT = 4, PC_OP_LT = 5 };
/* pc_eval_affinity inventory flags, one byte per row */
enum { PC_UNKNOWN_VALUE = 1, PC_UNKNOWN_KEY = 2 };
#define PC_LABEL_ABSENT 0xFFu   /* label value meaning "node does not carry this label" */
#define PC_ACTION_DROP 0xFFFFu  /* rule action: drop the packet */
#define PC_NO_PORT 0xFFFFu      /* pc_trace_out.last_port when not EGRESS */

/* terminal state of a trace */
enum { PC_EGRESS = 0, PC_DROP = 1, PC_MISS = 2, PC_TTL = 3 };

/* per-intent reason codes (low 7 bits); bit 7 = no compliant path exists */
enum {
    PC_R_PASS = 0,
    PC_R_NO_FEASIBLE_NODE = 1,
    PC_R_ENDPOINT_INFEASIBLE = 2,
    PC_R_NO_FLOW = 3,
    PC_R_LEAK = 4,
    PC_R_UNDELIVERED = 5,
    PC_R_WRONG_EGRESS = 6,
    PC_R_MALFORMED = 7,
    PC_R_FORBIDDEN_SWITCH = 8,   /* pc_report_paths only */
    PC_R_WAYPOINT_MISSED = 9,    /* pc_report_paths only */
    PC_R_NO_COMPLIANT_PATH = 0x80
};

/* sticky data-error bits */
enum {
    PC_DERR_PRED = 1,     /* a row references a predicate with label >= L, op > 2, a reserved field set,
                             or value 255 in an In/NotIn set */
    PC_DERR_OFFSETS = 2,  /* a CSR offset pair is negative, decreasing or past the array end */
    PC_DERR_ACTION = 4,   /* rule action (not DROP) >= number of ports of its switch */
    PC_DERR_SWITCH = 8,   /* switch / vertex id out of range (port peer, ingress, src, target) */
    PC_DERR_JUR = 16,     /* jurisdiction / region >= 32 */
    PC_DERR_GRAPH = 32,   /* adjacency entry out of [0, V) */
    PC_DERR_INTENT = 64,  /* intent record out of range or kind not in {1,2,3} */
    PC_DERR_NODE = 128    /* a listed node id outside [0, N) (pc_update_nodes) */
};

/* One selector predicate, 40 bytes.  vals is a 256-bit value set (bit v of
 * word v>>6); bit 255 must be clear (0xFF means absent).  Exists ignores vals. */
typedef struct pc_pred {
    uint16_t label;
    uint8_t op;
    uint8_t rsv0;     /* must be 0 */
    uint32_t rsv1;    /* must be 0 */
    uint64_t vals[4];
} pc_pred;

/* 104-bit 5-tuple, 16 bytes: w[0] src ip, w[1] dst ip, w[2] sport<<16 | dport,
 * w[3] proto in bits 0..7 (bits 8..31 zero by convention; they take part in
 * matching like any other bit). */
typedef struct pc_key {
    uint32_t w[4];
} pc_key;

/* One ternary flow rule, 40 bytes.  Matches header h iff ((h ^ value) & mask)
 * == 0 in all four words (mask bit 1 = care).  Larger priority wins; equal
 * priorities go to the lower index within the switch's table.  action is a
 * local out-port of the switch, or PC_ACTION_DROP. */
typedef struct pc_rule {
    pc_key value;
    pc_key mask;
    uint16_t priority;
    uint16_t action;
    uint32_t rsv;
} pc_rule;

/* Result of one trace, 12 bytes. */
typedef struct pc_trace_out {
    uint32_t jmask;       /* OR of 1<<jur[s] over every switch visited, ingress included */
    int32_t last_switch;  /* switch where the trace ended */
    uint16_t last_port;   /* egress port when state == PC_EGRESS, else PC_NO_PORT */
    uint8_t hops;         /* links crossed */
    uint8_t state;        /* PC_EGRESS / PC_DROP / PC_MISS / PC_TTL */
} pc_trace_out;

/* Expected egress of an intent's flows, 12 bytes (-1 = not checked). */
typedef struct pc_flow_expect {
    int32_t dst_switch;
    int32_t dst_port;
    int32_t reach_q;      /* index into the reach array, -1 = none */
} pc_flow_expect;

/* One intent, 32 bytes.  kind: bit 0 = compute check, bit 1 = network check
 * (1 compute, 2 network, 3 hybrid). */
typedef struct pc_intent {
    uint8_t kind;
    uint8_t pad[3];
    int32_t sel_row;      /* selector row (compute / hybrid) */
    int32_t src_node;     /* hybrid: nodes the endpoints were placed on */
    int32_t dst_node;
    int32_t trace_begin;  /* traces [trace_begin, trace_end) carry the intent's flows */
    int32_t trace_end;
    uint32_t allowed;     /* allowed jurisdictions, bit j = jurisdiction j */
    uint32_t pad2;
} pc_intent;

/* Path constraints of an intent's flows for pc_report_paths, 8 bytes: masks
 * over the watch slots of each of the intent's traces (pc_trace_flows_watch).
 * must: slots holding required waypoints; forbid: slots holding forbidden
 * switches. */
typedef struct pc_path_expect {
    uint32_t must;
    uint32_t forbid;
} pc_path_expect;

/* Verdict summary: counts[kind & 3][reason & 0x7F], no_path[kind & 3] counts
 * intents with PC_R_NO_COMPLIANT_PATH set. */
typedef struct pc_summary {
    uint64_t counts[4][16];
    uint64_t no_path[4];
} pc_summary;

typedef struct pc_ctx pc_ctx;

/* Create a context on HIP device `device`.  Returns PC_OK and *out, or
 * PC_EINVAL (bad device / NULL out) or PC_EDEVICE. */
int pc_create(pc_ctx **out, int device);

/* Free the context and its scratch.  Synchronises the device.  NULL is a no-op. */
int pc_destroy(pc_ctx *ctx);

/* Text of the last error on this context ("" if none).  Valid until the next call. */
const char *pc_last_error(const pc_ctx *ctx);

/* PC_VERSION of the library. */
int pc_version(void);

/* Synchronise `stream`, store the sticky data-error word in *flags (host
 * pointer) and clear it when `clear` is non-zero. */
int pc_data_errors(pc_ctx *ctx, void *stream, uint32_t *flags, int clear);

/* Per-kernel GPU timing, for benchmarks.  pc_profile(ctx, 1) resets the
 * tallies and brackets every library kernel launched on `ctx` afterwards
 * with HIP events on the launch's stream; pc_profile(ctx, 0) resets and
 * stops.  pc_profile_read waits for the recorded events and returns, for
 * the idx-th kernel name seen since the reset, the number of launches and
 * their summed duration in milliseconds (*name stays valid until the next
 * pc_profile call); PC_EINVAL when idx is past the last kernel. */
int pc_profile(pc_ctx *ctx, int enable);
int pc_profile_read(pc_ctx *ctx, int idx, const char **name, int64_t *launches, double *total_ms);

/* Measurement aid for the instruction-issue rooflines: times `reps`
 * launches (after one untimed) of a kernel that fills every wave slot with
 * eight independent dependency chains of one 32-bit integer VALU form and
 * touches no memory, and returns the wave-wide VALU instructions retired per
 * second in *wave_instr_per_s (the nominal peak is one per CU per clock).
 * op: 0 = v_add_u32 / v_sub_u32, 1 = v_xor_b32, 2 = v_and_or_b32 with three
 * vector sources, 3 = v_and_or_b32 with two vector sources and a scalar,
 * 4 = v_lshlrev_b64 by a scalar amount, 5 = v_add_u32 / v_sub_u32 in their
 * VOP3 encoding, 6 = s_xor_b32 (scalar ALU; the rate is then scalar
 * instructions per second), 7 = v_mov_b64, 8 = v_cmp_ne_u32 into scalar
 * register pairs, 9 = v_cndmask_b32 by a scalar register pair, 10 = v_bfi_b32,
 * 11 = v_xor_b32 with a scalar source, 12 = v_mov_b32, 13 = v_xor_b32 with an
 * inline constant, 14 = v_xor_b32 with a 32-bit literal.  When clock_hz is not NULL, the first wavefront of the last
 * timed launch reads the shader-clock and constant-rate counters around its
 * loop and *clock_hz receives the shader clock under that load (this path
 * allocates 16 bytes of device memory for the duration of the call).
 * Waits for its launches on `stream`.  PC_EINVAL for a NULL ctx or rate
 * output, reps < 1 or an op outside 0..14. */
int pc_measure_valu(pc_ctx *ctx, int op, int reps, double *wave_instr_per_s, double *clock_hz, void *stream);

/*
 * A1 -- placement constraints.  For every selector row i in [0, I) and node
 * n in [0, N): bit n of feasible[i] is set iff node n satisfies every
 * predicate of row i (an empty row admits every node):
 *   In S    : label present and its value in S
 *   NotIn S : label absent, or its value not in S
 *   Exists  : label present
 * labels   : uint8 [N][L], node-major; PC_LABEL_ABSENT = absent.
 * pred_off : int32 [I+1]; row i owns preds[pred_off[i] .. pred_off[i+1]).
 * preds    : pc_pred [n_preds].
 * feasible : uint64 [I][W], W = ceil(N/64); node n is bit n&63 of word n>>6;
 *            padding bits of the last word are written as 0.
 * popcnt   : uint32 [I], number of admitted nodes per row.
 * Limits: 0 <= N, 1 <= L <= 65535 (L = 0 allowed when no predicate exists),
 * 0 <= I, n_preds >= 0.  A malformed predicate admits no node
 * (PC_DERR_PRED); a malformed offset pair empties the row (PC_DERR_OFFSETS).
 */
int pc_eval_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L,
                      const int32_t *pred_off, const pc_pred *preds, int64_t n_preds, int32_t I,
                      uint64_t *feasible, uint32_t *popcnt, void *stream);

/*
 * pc_eval_selectors for callers that cannot allocate device memory: code
 * recorded into a HIP graph, tight serving loops, and hosts whose harness
 * forbids hipMalloc.  Same arguments, results, errors and data-error flags
 * as pc_eval_selectors; its scratch (value planes, compiled row programs,
 * popcount partials) lives in a fixed array of PC_NOALLOC_SCRATCH_BYTES that
 * the library's code object holds on each device until the process ends,
 * and the call makes no allocation (no hipMalloc / hipFree; with profiling
 * off, no event either).  A workload whose scratch would exceed the array
 * returns PC_EINVAL before any device work, naming the bytes it needs
 * (for N <= 8192 nodes the value planes take (L * min(N, 256) + 1) * 1152
 * bytes, each row 64 bytes and each predicate 16 bytes).  Every call on a
 * device shares that device's array: calls that overlap on one device (on
 * different streams or host threads, through any context) race and must be
 * ordered by the caller.
 */
#define PC_NOALLOC_SCRATCH_BYTES (64u << 20)
int pc_eval_selectors_noalloc(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                              const pc_pred *preds, int64_t n_preds, int32_t I, uint64_t *feasible, uint32_t *popcnt,
                              void *stream);

/*
 * A1, full node affinity -- placement directives compiled into Kubernetes
 * node selection criteria and affinity rules (paper: Intent Translation,
 * Service Placement Module), with the validator's cross-check of every
 * referenced label against the node-label inventory (Failure modes,
 * hallucinated identifiers).  Row i holds for node n iff at least one of
 * its terms holds; a term holds iff every one of its expressions holds.  A
 * row with no terms holds for every node; a term with no expressions holds
 * for none.  Operators: In, NotIn, Exists as in pc_eval_selectors, and
 *   DoesNotExist : label absent
 *   Gt / Lt      : label present and its value (0..254, the integer it
 *                  encodes) > / < t, t = (int64_t) vals[0]; vals[1..3] = 0.
 * labels   : uint8 [N][L], node-major; PC_LABEL_ABSENT = absent.
 * row_off  : int32 [I+1]; row i owns terms row_off[i] .. row_off[i+1].
 * term_off : int32 [n_terms+1]; term t owns preds[term_off[t] .. term_off[t+1]).
 * preds    : pc_pred [n_preds].
 * feasible : uint64 [I][W], W = ceil(N/64), as pc_eval_selectors.
 * popcnt   : uint32 [I].
 * unknown  : uint8 [I]; PC_UNKNOWN_VALUE when a well-formed In/NotIn
 *            expression of the row names a value no node carries for its
 *            label, PC_UNKNOWN_KEY when a well-formed expression names a
 *            label every node lacks (whether or not the expression holds).
 * All arrays are device memory owned by the caller.  Limits: 0 <= N,
 * 1 <= L <= 65535 (L = 0 allowed when no predicate exists), 0 <= I,
 * 0 <= n_terms, 0 <= n_preds.  Malformed data: an expression with label
 * >= L, op > 5, a reserved field set, value 255 in an In/NotIn set or
 * vals[1..3] != 0 for Gt/Lt holds for no node (PC_DERR_PRED, raised for
 * any such expression inside a term with a valid offset pair); a bad term
 * offset pair empties that term, a bad row offset pair the row
 * (PC_DERR_OFFSETS).
 */
int pc_eval_affinity(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *row_off,
                     int32_t I, const int32_t *term_off, int32_t n_terms, const pc_pred *preds, int64_t n_preds,
                     uint64_t *feasible, uint32_t *popcnt, uint8_t *unknown, void *stream);

/*
 * A1, preferred node affinity -- the secondary objective of placement:
 * among the configurations that satisfy an intent, one that is best for
 * secondary objectives (paper: Problem Definition, item 3), in the
 * Kubernetes form of weighted preferred terms (affinity rules of the
 * placement directives; Service Placement Module).  Row i owns the terms
 * row_off[i] .. row_off[i+1]; term t has weight weight[t] (1..100) and the
 * expressions term_off[t] .. term_off[t+1], which hold as in
 * pc_eval_affinity (all of them; a term with no expressions holds for no
 * node).  score(i, n) = sum of the weights of row i's terms that hold for
 * node n.  Among the row's feasible nodes the best node has the largest
 * score, the lowest index among equal scores.
 * labels     : uint8 [N][L], node-major; PC_LABEL_ABSENT = absent.
 * feasible   : uint64 [I][W], W = ceil(N/64), as written by pc_eval_affinity
 *              or pc_eval_selectors (bits past N are ignored); NULL = every
 *              node is feasible.
 * row_off    : int32 [I+1]; term_off : int32 [n_terms+1];
 * weight     : uint32 [n_terms]; preds : pc_pred [n_preds].
 * best_node  : int32 [I], the best feasible node, -1 when none is feasible.
 * best_score : uint32 [I], its score (0 when none).
 * n_best     : uint32 [I], the number of feasible nodes with that score (0
 *              when none).
 * All arrays are device memory owned by the caller.  Limits: 0 <= N,
 * 1 <= L <= 65535 (L = 0 allowed when no expression exists), 0 <= I,
 * 0 <= n_terms, 0 <= n_preds.  Malformed data: a weight outside 1..100 or
 * a malformed expression (as pc_eval_affinity) makes its term hold for no
 * node (PC_DERR_PRED, raised for any such term, and for any such
 * expression inside a term with a valid offset pair); a bad term offset
 * pair empties the term; a bad row offset pair or a row of more than
 * PC_PREF_MAX_TERMS terms leaves the row without terms, every score 0
 * (PC_DERR_OFFSETS).
 */
#define PC_PREF_MAX_TERMS 655
int pc_score_preferred(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const uint64_t *feasible,
                       const int32_t *row_off, int32_t I, const int32_t *term_off, int32_t n_terms,
                       const uint32_t *weight, const pc_pred *preds, int64_t n_preds, int32_t *best_node,
                       uint32_t *best_score, uint32_t *n_best, void *stream);

/*
 * A2+A3+A4 -- routing constraints on realised paths.  Each trace t starts at
 * switch ingress[t] with header hdr[t] and repeats: find the rule of
 * highest priority (ties: lower index) matching the header; none -> MISS;
 * DROP action -> DROP; a port whose peer is -1 faces a host -> EGRESS there;
 * a forward after `ttl` links -> TTL (the neighbour is not visited);
 * otherwise move to the peer switch.  jmask ORs 1<<jur[s] of every visited
 * switch.
 * port_off : int32 [S+1]; switch s owns ports port_off[s] .. port_off[s+1].
 * port_peer: int32 [n_ports]; peer switch of each port, -1 = host port.
 * jur      : uint8 [S], jurisdiction (< 32) of each switch.
 * rule_off : int32 [S+1]; switch s owns rules[rule_off[s] .. rule_off[s+1]).
 * rules    : pc_rule [n_rules].
 * hdr      : pc_key [T]; ingress: int32 [T]; out: pc_trace_out [T].
 * Limits: 0 <= S, 0 <= T, 0 <= ttl <= 255.  Malformed data: ingress or peer
 * out of range -> MISS (PC_DERR_SWITCH); invalid action -> MISS
 * (PC_DERR_ACTION); jur >= 32 adds no bit (PC_DERR_JUR); bad offsets -> the
 * switch has no rules / ports (PC_DERR_OFFSETS).
 */
int pc_trace_flows(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer,
                   int64_t n_ports, const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules,
                   int64_t n_rules, const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl,
                   pc_trace_out *out, void *stream);

/*
 * A5 -- compliant-path existence and hop distance.  For query q, vertex v is
 * allowed iff bit region[v] of allowed[q] is set; dist is the BFS hop
 * distance from src[q] inside the subgraph induced by the allowed vertices
 * of the undirected CSR graph, -1 if unreachable or if src[q] itself is not
 * allowed.
 * adj_off: int32 [V+1]; adj: int32 [n_adj]; region: uint8 [V].
 * src, allowed, target: [Q]; target may be NULL.
 * dist   : int32 [Q][V] (row-major) when target == NULL, else int32 [Q] with
 *          the distance to target[q].
 * Limits: 0 <= V, 0 <= Q.  Malformed: adj entry out of range is skipped
 * (PC_DERR_GRAPH); region >= 32 is never allowed (PC_DERR_JUR); src/target
 * out of range gives -1 (PC_DERR_SWITCH); bad offsets: no neighbours.
 */
int pc_masked_reach(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                    const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                    const int32_t *target, int32_t *dist, void *stream);

/*
 * A6 -- per-intent verdict.  compute (kind bit 0): popcnt[sel_row] > 0
 * (else NO_FEASIBLE_NODE); hybrid: both src_node and dst_node admitted by
 * the row (else ENDPOINT_INFEASIBLE).  network (kind bit 1): the trace range
 * is non-empty (else NO_FLOW, the no-op policy); every trace satisfies
 * jmask within allowed (else LEAK), state EGRESS (else UNDELIVERED), at
 * expect.dst_switch / dst_port when those are >= 0 (else WRONG_EGRESS).  The
 * reason is the smallest failing code (compute codes first); bit 7 is set
 * when expect.reach_q >= 0 and reach[reach_q] < 0.  A record pointing out of
 * range, or kind not in {1,2,3}: MALFORMED (PC_DERR_INTENT).
 * intents: pc_intent [I]; feasible: uint64 [rows][W]; popcnt: uint32 [rows];
 * N: number of nodes; traces: pc_trace_out [T]; expect: pc_flow_expect [I];
 * reach: int32 [Q].
 * pass   : uint64 [ceil(I/64)], bit i&63 of word i>>6 = intent i passes.
 * reason : uint8 [I].
 * summary: pc_summary (device memory), overwritten.
 */
int pc_report(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible,
              int32_t W, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
              const pc_flow_expect *expect, const int32_t *reach, int32_t Q, uint64_t *pass,
              uint8_t *reason, pc_summary *summary, void *stream);

/*
 * A2+A3, incremental re-validation after rule changes.  The paper's
 * validator re-checks continuously as the deployed state changes (abstract;
 * network state that changes with placement, Domain-specific performance).
 * A walk reads only the flow tables of the switches it visits, so when the
 * rules of some switches change, only traces whose walk visited one of
 * them can change.  Every trace carries a visited-switch summary: bit
 * (s mod 64) of vsum[t] for every switch s on its walk (ingress included;
 * 0 for an invalid ingress), and, when walk is not NULL, a walk record:
 * walk[t][0 .. 8) = the first 8 switches of its walk in order, -1 past its
 * end (all -1 for an invalid ingress).
 * C < 0  : trace every trace from scratch, as pc_trace_flows, and write
 *          vsum; *n_retraced = T.
 * C >= 0 : out[t] and vsum[t] hold the results of an earlier call on the
 *          same topology, headers, ingresses and ttl, and the tables
 *          passed now differ from those only in the rules of the switches
 *          changed[0 .. C) (table sizes may change).  A trace is traced
 *          again on the tables passed now, and its out / vsum / walk
 *          overwritten, when its walk record lists all of its walk
 *          (out[t].hops + 1 <= 8) and names a changed switch, or, for a
 *          longer walk or with walk NULL, when its vsum meets the bit of a
 *          changed switch; the others are left as they are.  The result
 *          equals a call with C < 0 on the tables passed now.
 *          *n_retraced = the number of traces traced again (exactly those
 *          that visited a changed switch when every walk fits its record;
 *          shared summary bits add others).
 * changed    : int32 [C]; ids outside [0, S) are ignored (PC_DERR_SWITCH),
 *              repeats are harmless.
 * out        : pc_trace_out [T], read and written.
 * vsum       : uint64 [T], read and written.
 * walk       : int32 [T][8], read and written, or NULL (selection by the
 *              summaries alone).  With C >= 0 the records must be those
 *              written with out / vsum: a call with walk NULL leaves them
 *              stale for later calls.
 * n_retraced : int32, device memory.
 * Prepared tables: by default every call prepares every switch's tables,
 * so the result depends only on the arguments.  After
 * pc_trace_keep_tables(ctx, 1) the context keeps the prepared tables of its
 * last pc_trace_flows_delta call, and a call with C >= 0 and the same S
 * reuses them, re-preparing only the changed switches, when no switch's
 * number of 32-rule groups changed (otherwise it prepares every switch).
 * That reuse is correct only under the caller's promise that the tables
 * passed differ from those of the context's previous pc_trace_flows_delta
 * call only in the changed switches' rules; the library does not check the
 * contents of unlisted switches.  A call with C < 0 always starts from a
 * full preparation.  Every call sweeps the whole input for data errors, as
 * pc_trace_flows (with reuse, the action flags of switches not re-prepared
 * are the ones found when they were prepared).
 */
/* Declare (enable = 1) or withdraw (enable = 0) the promise that, on this
 * context, consecutive pc_trace_flows_delta calls with C >= 0 pass tables
 * that differ from the previous call's only in the listed switches; with
 * it, those calls re-prepare only the listed switches (see above).
 * Withdrawing drops the kept tables.  Off on a new context.  PC_EINVAL on
 * a NULL context. */
int pc_trace_keep_tables(pc_ctx *ctx, int enable);

int pc_trace_flows_delta(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer,
                         int64_t n_ports, const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules,
                         int64_t n_rules, const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl,
                         const int32_t *changed, int32_t C, pc_trace_out *out, uint64_t *vsum, int32_t *walk,
                         int32_t *n_retraced, void *stream);

/*
 * Waypoint and forbidden-switch constraints on realised paths.  The paper's
 * routing constraints name required waypoints and forbidden vertices (Formal
 * Model and Satisfaction, "Configuration"; the must_go / forbidden lists of
 * the JSON constraints in "Network orchestration"), and a network check
 * asserts that every realised path of a flow avoids the forbidden switches
 * and includes the required waypoints (Automated Validation Pipeline,
 * validator check definition).
 *
 * pc_trace_flows_watch: pc_trace_flows, and in addition, for every trace t,
 * bit k of visit[t] is set iff the trace visited switch watch[t][k] at any
 * point of its walk (ingress and last switch included).  Neighbours that a
 * TTL-terminated trace would have moved to are not visited.
 * watch : int32 [T][K], row-major; -1 = an unused slot (never matches).
 * K     : slots per trace, 0 <= K <= 32 (K = 0: watch may be NULL and every
 *         visit word is 0).
 * visit : uint32 [T], written for every trace.
 * Malformed: a watch entry < -1 or >= S matches nothing (PC_DERR_SWITCH).
 */
int pc_trace_flows_watch(pc_ctx *ctx, int32_t S, const int32_t *port_off, const int32_t *port_peer,
                         int64_t n_ports, const uint8_t *jur, const int32_t *rule_off, const pc_rule *rules,
                         int64_t n_rules, const pc_key *hdr, const int32_t *ingress, int32_t T, int32_t ttl,
                         const int32_t *watch, int32_t K, pc_trace_out *out, uint32_t *visit, void *stream);

/*
 * pc_masked_reach_via: length of the shortest walk src[q] -> via[q][0] ->
 * ... -> via[q][m-1] -> target[q] that stays on allowed switches (bit
 * region[v] of allowed[q], as in pc_masked_reach) none of which is in
 * forbid[q]; m is the number of via entries before the first -1.  Each leg
 * is a shortest path of the induced subgraph, so the walk may repeat
 * switches.  dist[q] = the sum of the leg distances, or -1 when any leg has
 * no path (including an endpoint or waypoint that is not allowed or is
 * forbidden).
 * via   : int32 [Q][Kv] row-major (Kv >= 0; NULL when Kv == 0).
 * forbid: int32 [Q][Kf] row-major, -1 = unused slot (Kf >= 0; NULL when
 *         Kf == 0).
 * target: int32 [Q] (required).  dist: int32 [Q].
 * Limits: 0 <= Kv, Kf <= 32.  Malformed: a via or forbid entry < -1 or >= V
 * raises PC_DERR_SWITCH; such a waypoint has no path, such a forbidden entry
 * is ignored.  Scratch: int32 [Q][Kv + 1] leg records.
 */
int pc_masked_reach_via(pc_ctx *ctx, int32_t V, const int32_t *adj_off, const int32_t *adj, int64_t n_adj,
                        const uint8_t *region, int32_t Q, const int32_t *src, const uint32_t *allowed,
                        const int32_t *target, const int32_t *via, int32_t Kv, const int32_t *forbid,
                        int32_t Kf, int32_t *dist, void *stream);

/*
 * pc_report_paths: pc_report with the path checks of network intents added.
 * A trace whose visit word meets pexp[i].forbid fails with
 * PC_R_FORBIDDEN_SWITCH; one whose visit word lacks a bit of pexp[i].must
 * fails with PC_R_WAYPOINT_MISSED.  Per trace the smallest failing code
 * counts, as for the other trace codes (so LEAK, UNDELIVERED and
 * WRONG_EGRESS come first).
 * visit: uint32 [T] (pc_trace_flows_watch); pexp: pc_path_expect [I].
 */
int pc_report_paths(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible,
                    int32_t W, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
                    const pc_flow_expect *expect, const int32_t *reach, int32_t Q, const uint32_t *visit,
                    const pc_path_expect *pexp, uint64_t *pass, uint8_t *reason, pc_summary *summary,
                    void *stream);

/*
 * NEXT-4 -- verdict-only runs.  The verdict (pc_report) reads each selector
 * row's popcount and, for hybrid intents, two placed endpoints' bits (paper:
 * an intent passes only if all of its checks pass; hybrid endpoints are the
 * nodes the pods were placed on).  These three calls give it both without
 * materialising the I x ceil(N/64) bitset.
 *
 * pc_eval_selectors_count: popcnt exactly as pc_eval_selectors, no bitset.
 * pc_probe_selectors: bit[k] = 1 iff node probe_node[k] satisfies selector
 *   row probe_row[k]; 0 when the row is outside [0, I) or the node outside
 *   [0, N) (PC_DERR_NODE).  probe_row, probe_node: int32 [P]; bit: uint8 [P].
 * pc_report_counts: pc_report with each hybrid intent i's endpoint bits read
 *   from ends[2i] (src_node) and ends[2i + 1] (dst_node), bit 0 of each,
 *   instead of bitset words; ends: uint8 [2I] (entries of non-hybrid intents
 *   are not read).
 * Arguments, layouts, limits and malformed-data handling otherwise as
 * pc_eval_selectors / pc_report.
 */
int pc_eval_selectors_count(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                            const pc_pred *preds, int64_t n_preds, int32_t I, uint32_t *popcnt, void *stream);
int pc_probe_selectors(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                       const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *probe_row,
                       const int32_t *probe_node, int32_t P, uint8_t *bit, void *stream);
int pc_report_counts(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint32_t *popcnt,
                     int32_t N, const uint8_t *ends, const pc_trace_out *traces, int32_t T,
                     const pc_flow_expect *expect, const int32_t *reach, int32_t Q, uint64_t *pass, uint8_t *reason,
                     pc_summary *summary, void *stream);

/* Most nodes one pc_update_nodes call accepts. */
#define PC_UPDATE_MAX_NODES 4096

/*
 * NEXT-4 -- continuous re-validation: incremental re-evaluation of selector
 * rows after the labels of some nodes changed (paper, Abstract: continuous
 * cross-layer compliance checking).  labels already holds the new labels;
 * feasible / popcnt hold pc_eval_selectors' output for labels that differ
 * from these only at nodes[0..M).  Afterwards they hold pc_eval_selectors'
 * output for the new labels: for every row and every listed node the row's
 * bit of the node is set to the selector definition on its new labels, and
 * the row's popcount moves by the change.  Repeated nodes are allowed.
 * Arguments and layouts as pc_eval_selectors; nodes: int32 [M] device
 * array.  Limits: 0 <= M <= PC_UPDATE_MAX_NODES.  Malformed data: a listed
 * node outside [0, N) is skipped (PC_DERR_NODE); rows and predicates as in
 * pc_eval_selectors (PC_DERR_OFFSETS, PC_DERR_PRED).  The incremental cost
 * grows with the number of distinct bitset words the nodes touch per row;
 * above W / 32 listed nodes the call evaluates every row in full instead
 * (the same result; environment variable PC_UPDATE_FULL_ABOVE overrides the
 * threshold).
 */
int pc_update_nodes(pc_ctx *ctx, const uint8_t *labels, int32_t N, int32_t L, const int32_t *pred_off,
                    const pc_pred *preds, int64_t n_preds, int32_t I, const int32_t *nodes, int32_t M,
                    uint64_t *feasible, uint32_t *popcnt, void *stream);

/* Largest topology pc_synthesize_paths accepts (its per-request search
 * state lives in on-chip memory). */
#define PC_SYNTH_MAX_V 12288

/*
 * NEXT-2 -- compliant path synthesis (paper: Network orchestration -- a path
 * scheduler performs graph search over the current topology, weighted
 * Dijkstra with a BFS fallback, to produce a path that respects the
 * constraints; each path is transformed into per-hop flow rules).
 * Graph: switch s owns ports port_off[s] .. port_off[s+1]; a port with peer
 * v in [0, V) and weight >= 1 is a link s -> v (weight NULL: every link
 * weighs 1, i.e. BFS).  A switch is usable by request q when its region is
 * allowed by allowed[q] and it is not in forbid[q][0..Kf) (-1 = unused).
 * The walk of request q is src[q] -> via[q][0] -> ... -> target[q] (the
 * waypoint list ends at its first -1), one minimum-weight leg per stop
 * through usable switches; the predecessor of every switch on a leg is the
 * lowest-numbered u with a link u -> v and dist(u) + w = dist(v).
 * Outputs (caller-owned device arrays):
 *   hops  : int32 [Q], links of the walk, -1 when the request fails.
 *   path  : int32 [Q][max_hops + 1], the walk's switches (src first), -1 past
 *           its end (all -1 on failure).
 *   rules : pc_rule [Q][max_hops + 1], one per switch of the walk: value =
 *           key[q], mask = the 104 key bits (words 0-2 and bits 0-7 of word
 *           3), priority = prio, action = the switch's port of least (weight,
 *           index) to the next switch, out_port[q] at the last switch; zero
 *           past the walk's end (all zero on failure).  A walk that passes a
 *           switch twice cannot be realised by rules that match the 5-tuple
 *           only; it is returned as found.
 * A request fails when an endpoint or waypoint is out of range or not
 * usable, a leg has no path, out_port[q] is not a port of the target, or the
 * walk has more than max_hops links.  Distances are sums of link weights
 * below 2^31 - 1: a switch whose minimum distance from the leg's start is
 * 2^31 - 1 or more counts as unreachable.
 * Limits: 0 <= V <= PC_SYNTH_MAX_V, 0 <= Q, 0 <= Kv, Kf <= 32,
 * 0 <= max_hops <= 255, 0 <= prio <= 65535.  Malformed data: bad port_off
 * pair -> the switch has no ports (PC_DERR_OFFSETS); peer < -1 or >= V, src
 * or target outside [0, V), via / forbid entry < -1 or >= V
 * (PC_DERR_SWITCH); region >= 32 never allowed (PC_DERR_JUR); a zero weight
 * -> that port is no link (PC_DERR_GRAPH); out_port not a port of a target
 * with valid offsets (PC_DERR_ACTION).
 */
int pc_synthesize_paths(pc_ctx *ctx, int32_t V, const int32_t *port_off, const int32_t *port_peer,
                        int64_t n_ports, const uint32_t *weight, const uint8_t *region, int32_t Q,
                        const int32_t *src, const int32_t *target, const uint32_t *allowed, const int32_t *via,
                        int32_t Kv, const int32_t *forbid, int32_t Kf, const pc_key *key, const int32_t *out_port,
                        int32_t prio, int32_t max_hops, int32_t *hops, int32_t *path, pc_rule *rules, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PC_H */
