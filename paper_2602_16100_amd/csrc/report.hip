// A6 -- per-intent verdict.  An intent passes only if every one of its
// validator checks passes (Automated Validation Pipeline, validator check
// definition); an intent that cannot be enforced fails closed (the
// "unenforceable" computing example; failure modes "Ambiguous path
// specification" -> no-op policy and "Hallucinated identifiers" -> no
// feasible node).  Reason codes and their order are the ones in pc.h.
//
// One thread per intent; pass bits are ballot-packed (one 64-bit word per
// wavefront); the (kind, reason) summary is reduced in LDS and added once
// per workgroup.  With visit words and path expectations (pc_report_paths),
// a network intent's traces must also avoid its forbidden switches and pass
// its required waypoints (the paper's Configuration: required waypoints,
// forbidden vertices; validator check definition).
#include "pc_internal.h"

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void k_report(int32_t I, const pc_intent *__restrict__ intents, int32_t rows,
                                                     const uint64_t *__restrict__ feasible, int32_t W,
                                                     const uint8_t *__restrict__ ends,
                                                     const uint32_t *__restrict__ popcnt, int32_t N,
                                                     const pc_trace_out *__restrict__ traces, int32_t T,
                                                     const pc_flow_expect *__restrict__ expect,
                                                     const int32_t *__restrict__ reach, int32_t Q,
                                                     const uint32_t *__restrict__ visit,
                                                     const pc_path_expect *__restrict__ pexp,
                                                     uint64_t *__restrict__ pass, uint8_t *__restrict__ reason,
                                                     unsigned long long *__restrict__ summary,
                                                     uint32_t *__restrict__ d_err)
{
    constexpr int kHist = 4 * 16 + 4;
    __shared__ unsigned int hist[kHist];
    const int tid = threadIdx.x, lane = tid & 63;
    if (tid < kHist) hist[tid] = 0;
    __syncthreads();
    const int32_t i = blockIdx.x * kThreads + tid;
    bool ok = false, bad = false;
    if (i < I) {
        const pc_intent it = intents[i];
        const pc_flow_expect ex = expect[i];
        const int kind = it.kind;
        bool malformed = kind < 1 || kind > 3;
        if (!malformed && (kind & 1)) {
            if (it.sel_row < 0 || it.sel_row >= rows) malformed = true;
            if (kind == 3 && (it.src_node < 0 || it.src_node >= N || it.dst_node < 0 || it.dst_node >= N))
                malformed = true;
        }
        if (!malformed && (kind & 2)) {
            if (it.trace_begin < 0 || it.trace_end < it.trace_begin || it.trace_end > T) malformed = true;
            if (ex.reach_q < -1 || ex.reach_q >= Q) malformed = true;
        }
        int r = 0;
        bool nopath = false;
        if (malformed) {
            r = PC_R_MALFORMED;
            bad = true;
        } else {
            if (kind & 1) {
                if (popcnt[it.sel_row] == 0) {
                    r = PC_R_NO_FEASIBLE_NODE;
                } else if (kind == 3) {
                    bool a, b;
                    if (feasible) {
                        const uint64_t *row = feasible + static_cast<int64_t>(it.sel_row) * W;
                        a = (row[it.src_node >> 6] >> (it.src_node & 63)) & 1;
                        b = (row[it.dst_node >> 6] >> (it.dst_node & 63)) & 1;
                    } else {  // endpoint bits from probes (verdict-only runs)
                        a = ends[2 * static_cast<int64_t>(i)] & 1;
                        b = ends[2 * static_cast<int64_t>(i) + 1] & 1;
                    }
                    if (!(a && b)) r = PC_R_ENDPOINT_INFEASIBLE;
                }
            }
            if (kind & 2) {
                if (r == 0) {
                    if (it.trace_end == it.trace_begin) r = PC_R_NO_FLOW;
                    const pc_path_expect pe = pexp ? pexp[i] : pc_path_expect{0u, 0u};
                    for (int32_t t = it.trace_begin; t < it.trace_end; ++t) {
                        const pc_trace_out tr = traces[t];
                        const uint32_t vis = visit ? visit[t] : 0u;
                        int code = 0;
                        if (tr.jmask & ~it.allowed) code = PC_R_LEAK;
                        else if (tr.state != PC_EGRESS) code = PC_R_UNDELIVERED;
                        else if ((ex.dst_switch >= 0 && tr.last_switch != ex.dst_switch) ||
                                 (ex.dst_port >= 0 && tr.last_port != ex.dst_port))
                            code = PC_R_WRONG_EGRESS;
                        else if (vis & pe.forbid) code = PC_R_FORBIDDEN_SWITCH;
                        else if ((vis & pe.must) != pe.must) code = PC_R_WAYPOINT_MISSED;
                        if (code && (r == 0 || code < r)) r = code;
                    }
                }
                if (ex.reach_q >= 0 && reach[ex.reach_q] < 0) nopath = true;
            }
        }
        reason[i] = static_cast<uint8_t>(r | (nopath ? PC_R_NO_COMPLIANT_PATH : 0));
        ok = r == 0;
        atomicAdd(&hist[(kind & 3) * 16 + r], 1u);
        if (nopath) atomicAdd(&hist[64 + (kind & 3)], 1u);
    }
    const uint64_t word = __ballot(ok);
    const int32_t i0 = i - lane;
    if (lane == 0 && i0 < I) pass[i0 >> 6] = word;
    if (__ballot(bad) && lane == 0) atomicOr(d_err, PC_DERR_INTENT);
    __syncthreads();
    if (tid < kHist && hist[tid]) atomicAdd(&summary[tid], static_cast<unsigned long long>(hist[tid]));
}

}  // namespace

int run_report(pc_ctx *ctx, int32_t I, const pc_intent *intents, int32_t rows, const uint64_t *feasible, int32_t W,
               const uint8_t *ends, const uint32_t *popcnt, int32_t N, const pc_trace_out *traces, int32_t T,
               const pc_flow_expect *expect, const int32_t *reach, int32_t Q, const uint32_t *visit,
               const pc_path_expect *pexp, uint64_t *pass, uint8_t *reason, pc_summary *summary, hipStream_t stream)
{
    static_assert(sizeof(pc_summary) == 68 * 8, "summary layout");
    launch_fill_u64(reinterpret_cast<uint64_t *>(summary), 68, 0, stream);
    PC_LAUNCH_CHECK(ctx);
    if (I == 0) return PC_OK;
    PC_TIMED(ctx, "k_report", stream, hipLaunchKernelGGL(k_report, dim3(static_cast<unsigned>((I + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                       stream, I, intents, rows, feasible, W, ends, popcnt, N, traces, T, expect, reach, Q, visit, pexp, pass, reason,
                       reinterpret_cast<unsigned long long *>(summary), ctx->d_err));
    PC_LAUNCH_CHECK(ctx);
    return PC_OK;
}
