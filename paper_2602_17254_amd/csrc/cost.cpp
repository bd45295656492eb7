// The congestion-aware cost model of Sec. 2.1, evaluated for a plan (host only).
//
// C(m, A) = steps(A) alpha + sum_k beta m_k c_k: each pass pays the start-up latency alpha, and its
// transmission lasts as long as its busiest directed link needs, beta times the bytes of every
// message that crosses that link (m_k c_k for chunks of one size). In a Trivance pass every rank
// of collective c sends one message towards each side along its active dimension, over the
// collective's distance; with the same size for every rank (the schedule is the same up to a
// shift), each directed link of that dimension carries `distance` such messages per collective.
// The bytes of a link direction are therefore sum over the collectives on that dimension of
// (message bytes x distance), and the busiest link is the largest of these over the dimensions
// and both directions.
//
// Message sizes (m bytes per rank, D collectives on m / D each, blocks of m / (n D)):
//   latency-optimal   the whole segment, m / D (Sec. 4.2); on sides that are not powers of three,
//                     one segment per distinct partial the receiver takes from the sender;
//   bandwidth-optimal n / 3^(t+1) blocks at reduce-scatter and all-gather step t (Sec. 4.1 and the
//                     closed form of Sec. 4.3; Lemma 1);
//   tree steps        per direction, the offsets of the active dimension's tree that forward
//                     that way in the step, times the not-yet-forwarded offsets of every other
//                     dimension, in blocks (Sec. 4.4); an all-gather step sends the same blocks
//                     back, so its directions swap.
#include <algorithm>

#include "plan.h"

namespace {

// Busiest directed link of one pass, in bytes per byte of m.
double pass_peak(const trivance_plan_t* p, const trivance::Pass& ps) {
    const double seg = 1.0 / p->D;  // a collective's share of m
    double load[trivance::kMaxDims][2] = {};
    for (int c = 0; c < p->D; ++c) {
        const int a = ps.dim[c];
        const double hops = ps.distance[c];
        double plus = 0.0, minus = 0.0;  // bytes of one rank's message towards + and -
        if (ps.phase == TRIVANCE_PHASE_LATENCY && !p->slots.empty()) {
            // slot programs: a message carries every distinct slot its receiver takes from it
            const trivance::SlotPass& sp = p->slots[&ps - p->passes.data()];
            bool to_plus[trivance::kMaxSlots] = {}, to_minus[trivance::kMaxSlots] = {};
            for (int i = 0; i < sp.nout[c]; ++i) {
                if (sp.left[c][i] >= 0) to_plus[sp.left[c][i]] = true;
                if (sp.right[c][i] >= 0) to_minus[sp.right[c][i]] = true;
            }
            for (int i = 0; i < sp.nin[c]; ++i) {
                plus += to_plus[i] ? seg : 0.0;
                minus += to_minus[i] ? seg : 0.0;
            }
        } else if (ps.phase == TRIVANCE_PHASE_LATENCY) {
            plus = minus = seg;
        } else if (!p->tree) {
            plus = minus = seg * (double)ps.kept_per_rank / p->n;
        } else {
            const trivance::DimTree& t = p->trees[a];
            double from_left = 0, from_right = 0;  // children moving towards + / towards -
            for (uint32_t e : t.recv[ps.dim_step[c]]) {
                if (e & trivance::kFromLeft) from_left += 1;
                if (e & trivance::kFromRight) from_right += 1;
            }
            double others = 1.0;
            for (int d = 0; d < p->D; ++d)
                if (d != a) others *= (double)p->trees[d].alive[ps.taken[c][d]].size();
            const double blk = seg / p->n;
            const bool rs = ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER;
            plus = blk * others * (rs ? from_left : from_right);
            minus = blk * others * (rs ? from_right : from_left);
        }
        load[a][0] += plus * hops;
        load[a][1] += minus * hops;
    }
    double peak = 0.0;
    for (int d = 0; d < p->D; ++d) peak = std::max(peak, std::max(load[d][0], load[d][1]));
    return peak;
}

}  // namespace

extern "C" int trivance_cost_model(const trivance_plan_t* plan, double bytes_per_rank, double alpha,
                                   double beta, double* pass_link_bytes, int pass_len,
                                   trivance_cost_result* out) {
    if (!plan || !out || !(bytes_per_rank >= 0.0) || !(alpha >= 0.0) || !(beta >= 0.0))
        return TRIVANCE_EINVAL;
    if (plan->variant == TRIVANCE_BRUCK_REF) return TRIVANCE_EUNSUPPORTED;
    const int P = (int)plan->passes.size();
    if (pass_link_bytes && pass_len < P) return TRIVANCE_ESIZE;
    double sum = 0.0;
    for (int i = 0; i < P; ++i) {
        const double peak = pass_peak(plan, plan->passes[i]);
        if (pass_link_bytes) pass_link_bytes[i] = peak * bytes_per_rank;
        sum += peak;
    }
    out->passes = P;
    out->latency = P * alpha;
    out->transmission = beta * bytes_per_rank * sum;
    out->total = out->latency + out->transmission;
    out->theta = sum * plan->D;
    return TRIVANCE_OK;
}
