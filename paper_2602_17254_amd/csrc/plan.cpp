// Host-side schedule generator and byte accounting of the emulated Trivance AllReduce.
//
// Steps and peers: Sec. 4.1 (pi(r, k) = r -/+ 3^k), Theorem 1 (log3 n steps), Sec. 4.2 (the
// latency-optimal variant uses the same pattern), Sec. 5 (one collective per torus dimension on
// 1/D of the data, switching dimension every step; Appendix B's index t = d + D k fixes the
// per-dimension step k = t div D). Unequal sides (rectangular tori) are not covered by Sec. 5;
// the rule used for them: collective c at global step t takes the first dimension, in cyclic
// order from (c + t) mod D, in which it still has steps left. With equal sides this is exactly
// (c + t) mod D at distance 3^(t div D). Block sets: the closed form of Sec. 4.3 says that the blocks
// forwarded to peer p at step k are p + sum_{i>k} e_i 3^i; equivalently the blocks a rank keeps
// after step k are those congruent to it modulo 3^(k+1). On a torus that congruence holds per
// dimension, with the exponent counting the steps taken so far in that dimension.
#include <cmath>
#include <cstdlib>
#include <new>

#include "plan.h"

using trivance::kGranule;
using trivance::kMaxDims;
using trivance::Pass;

namespace {

int log3_exact(int v) {
    int s = 0;
    long long m = 1;
    while (m < v) {
        m *= 3;
        ++s;
    }
    return m == v ? s : -1;
}

int ipow3(int e) {
    int v = 1;
    for (int i = 0; i < e; ++i) v *= 3;
    return v;
}

// Per collective: the dimension and distance of every global step, and the per-dimension
// moduli 3^(steps taken so far in that dimension) after every step.
struct Rotation {
    int dim[64][kMaxDims];
    int dist[64][kMaxDims];
    int modulus[64][kMaxDims][kMaxDims];
};

void fill_rotation(const trivance_plan_t* p, const int* steps_per_dim, Rotation* rot) {
    for (int c = 0; c < p->D; ++c) {
        int count[kMaxDims] = {};
        for (int t = 0; t < p->S; ++t) {
            int d = (c + t) % p->D;
            for (int i = 0; i < p->D; ++i) {
                const int cand = (c + t + i) % p->D;
                if (count[cand] < steps_per_dim[cand]) {
                    d = cand;
                    break;
                }
            }
            rot->dim[t][c] = d;
            rot->dist[t][c] = ipow3(count[d]);
            count[d] += 1;
            for (int dd = 0; dd < kMaxDims; ++dd)
                rot->modulus[t][c][dd] = dd < p->D ? ipow3(count[dd]) : 1;
        }
    }
}

Pass make_pass(const trivance_plan_t* p, const Rotation& rot, int phase, int t) {
    Pass ps{};
    ps.phase = phase;
    ps.step = t;
    for (int c = 0; c < kMaxDims; ++c) {
        ps.dim[c] = c < p->D ? rot.dim[t][c] : 0;
        ps.distance[c] = c < p->D ? rot.dist[t][c] : 1;
        for (int d = 0; d < kMaxDims; ++d) ps.modulus[c][d] = c < p->D ? rot.modulus[t][c][d] : 1;
    }
    ps.kept_per_rank = p->n / ipow3(t + 1);
    return ps;
}

// ---- sides that are not powers of three (Sec. 4.4) ----
//
// A ring (or torus dimension) of side n with 3^f < n < 3^(f+1) takes f full steps at distances
// 3^0..3^(f-1), then a final step at d = ceil((n - 3^f) / 2). Every block j is reduced along one
// tree so that each rank forwards each block once (Sec. 4.4); the tree is read from three
// ordinary Trivance trees rooted at offsets 0, +d and -d from j (offsets in (-n/2, n/2]): ranks
// beyond j's window (|offset| > R = (3^f - 1)/2) start in the tree of their side; then, until
// nothing changes, every rank on the path of a +/- member joins that tree, and a member of j's
// tree whose path meets another tree joins it. The root offsets +d and -d hand their partials
// to j in the final step. For n = 3^f this is the ordinary tree (d = 0, all offsets in j's
// window): an offset sends at the step of its lowest non-zero balanced-ternary digit.

// Balanced-ternary digits of v (lowest first, f of them); false if v needs more digits.
bool balanced_digits(long v, int f, int* e) {
    for (int i = 0; i < f; ++i) {
        const int r = (int)(((v % 3) + 3) % 3);
        e[i] = r == 2 ? -1 : r;
        v = (v - e[i]) / 3;
    }
    return v == 0;
}

int build_dim_tree(int n, trivance::DimTree* t) {
    t->side = n;
    if (n == 1) {
        t->S = 0;
        t->alive.assign(1, std::vector<uint32_t>(1, 0u));
        return TRIVANCE_OK;
    }
    int f = 0;
    long pw = 1;
    while (pw * 3 <= n) {
        pw *= 3;
        ++f;
    }
    const long R = (pw - 1) / 2;
    const long d = (n - pw + 1) / 2;
    const long lo = -((n - 1) / 2);
    auto canon = [&](long o) {
        long r = (o - lo) % n;
        if (r < 0) r += n;
        return r + lo;
    };
    auto idx = [&](long o) { return (size_t)(canon(o) - lo); };
    std::vector<int> fam(n);
    for (long o = lo; o < lo + n; ++o) fam[idx(o)] = o > R ? 1 : (o < -R ? -1 : 0);
    // offset of rank o relative to the root of tree `side`, if o lies in that tree's window
    auto rel_in = [&](long o, int side, long* rel) {
        const long cands[3] = {o, o + n, o - n};
        for (long c : cands) {
            const long r = c - side * d;
            if (r >= -R && r <= R) {
                *rel = r;
                return true;
            }
        }
        return false;
    };
    int e[32];
    for (int guard = 0;; ++guard) {
        if (guard > 4 * n + 8) return TRIVANCE_EUNSUPPORTED;
        bool changed = false;
        for (long o = lo; o < lo + n; ++o) {
            const int side = fam[idx(o)];
            long rel;
            if (!rel_in(o, side, &rel) || !balanced_digits(rel, f, e)) return TRIVANCE_EUNSUPPORTED;
            long pos = rel;
            long pw_i = 1;
            for (int i = 0; i < f; ++i, pw_i *= 3) {
                pos -= e[i] * pw_i;
                const long q = canon(pos + side * d);
                if (side != 0 && fam[idx(q)] != side) {
                    if (fam[idx(q)] != 0 || q == 0) return TRIVANCE_EUNSUPPORTED;
                    fam[idx(q)] = side;
                    changed = true;
                }
                if (side == 0 && fam[idx(q)] != 0) {
                    fam[idx(o)] = fam[idx(q)];
                    changed = true;
                    break;
                }
            }
        }
        if (!changed) break;
    }
    if (fam[idx(0)] != 0) return TRIVANCE_EUNSUPPORTED;

    // send step, direction and parent of every offset; receivers per step
    const int S = d ? f + 1 : f;
    std::vector<int> step(n, S), dir(n, 0);
    std::vector<long> parent(n, 0);
    for (long o = lo; o < lo + n; ++o) {
        if (o == 0) continue;
        const int side = fam[idx(o)];
        long rel = 0;
        if (!rel_in(o, side, &rel) || !balanced_digits(rel, f, e)) return TRIVANCE_EUNSUPPORTED;
        int k = f;
        int ek = side;
        long pw_k = 1;
        for (int i = 0; i < f; ++i, pw_k *= 3) {
            if (e[i] != 0) {
                k = i;
                ek = e[i];
                break;
            }
        }
        if (k >= S) return TRIVANCE_EUNSUPPORTED;
        const long dist = k < f ? pw_k : d;
        step[idx(o)] = k;
        dir[idx(o)] = ek;
        parent[idx(o)] = canon(o - ek * dist);
    }
    t->S = S;
    t->dist.assign(S, 0);
    t->dirs.assign(S, 0);
    t->recv.assign(S, std::vector<uint32_t>());
    t->alive.assign(S + 1, std::vector<uint32_t>());
    for (int k = 0; k < S; ++k) t->dist[k] = k < f ? ipow3(k) : (int)d;
    std::vector<std::vector<uint32_t>> flags(S, std::vector<uint32_t>(n, 0));
    for (long o = lo; o < lo + n; ++o) {
        if (o == 0) continue;
        const int k = step[idx(o)];
        const long par = parent[idx(o)];
        if (par != 0 && step[idx(par)] <= k) return TRIVANCE_EUNSUPPORTED;  // not a tree
        flags[k][idx(par)] |= dir[idx(o)] > 0 ? trivance::kFromRight : trivance::kFromLeft;
        t->dirs[k] |= dir[idx(o)] > 0 ? 2 : 1;
    }
    for (long o = lo; o < lo + n; ++o) {
        const uint32_t res = (uint32_t)((o % n + n) % n);
        for (int m = 0; m <= step[idx(o)]; ++m) t->alive[m].push_back(res);
        for (int k = 0; k < S; ++k)
            if (flags[k][idx(o)]) t->recv[k].push_back(res | flags[k][idx(o)]);
    }
    return TRIVANCE_OK;
}

// Tree plan: one tree per dimension; collective c at global step t takes the first dimension,
// in cyclic order from (c + t) mod D, in which it still has steps left (the rule used for
// unequal sides). Reduce-scatter passes t = 0..S-1, then the all-gather in reverse order.
int build_tree_plan(trivance_plan_t* p) {
    p->trees.assign(p->D, trivance::DimTree());
    p->S = 0;
    for (int dd = 0; dd < p->D; ++dd) {
        const int rc = build_dim_tree(p->dims[dd], &p->trees[dd]);
        if (rc != TRIVANCE_OK) return rc;
        p->S += p->trees[dd].S;
    }
    if (2 * p->S > 40) return TRIVANCE_EUNSUPPORTED;
    std::vector<Pass> rs(p->S);
    for (int t = 0; t < p->S; ++t) {
        rs[t] = Pass{};
        rs[t].phase = TRIVANCE_PHASE_REDUCE_SCATTER;
        rs[t].step = t;
        for (int c = 0; c < kMaxDims; ++c) {
            rs[t].distance[c] = 1;
            for (int dd = 0; dd < kMaxDims; ++dd) rs[t].modulus[c][dd] = 1;
        }
    }
    for (int c = 0; c < p->D; ++c) {
        int count[kMaxDims] = {};
        for (int t = 0; t < p->S; ++t) {
            int dsel = -1;
            for (int i = 0; i < p->D && dsel < 0; ++i) {
                const int cand = (c + t + i) % p->D;
                if (count[cand] < p->trees[cand].S) dsel = cand;
            }
            Pass& ps = rs[t];
            ps.dim[c] = dsel;
            ps.dim_step[c] = count[dsel];
            ps.distance[c] = p->trees[dsel].dist[count[dsel]];
            for (int dd = 0; dd < p->D; ++dd) ps.taken[c][dd] = count[dd];
            count[dsel] += 1;
        }
    }
    // every pass's offset lists must fit the kernel-argument table
    for (int t = 0; t < p->S; ++t) {
        size_t entries = 0;
        for (int c = 0; c < p->D; ++c)
            for (int dd = 0; dd < p->D; ++dd)
                entries += dd == rs[t].dim[c]
                               ? p->trees[dd].recv[rs[t].dim_step[c]].size()
                               : p->trees[dd].alive[rs[t].taken[c][dd]].size();
        if (entries > (size_t)trivance::kMaxTab) return TRIVANCE_EUNSUPPORTED;
    }
    for (int t = 0; t < p->S; ++t) p->passes.push_back(rs[t]);
    for (int t = p->S - 1; t >= 0; --t) {
        Pass ps = rs[t];
        ps.phase = TRIVANCE_PHASE_ALLGATHER;
        p->passes.push_back(ps);
    }
    p->tree = true;
    return TRIVANCE_OK;
}

// ---- latency-optimal variant on sides that are not powers of three (Sec. 4.2 with Sec. 4.4) ----
//
// A rank keeps partial sums ("slots") over boxes of offsets relative to itself (one interval per
// dimension). The result is the whole torus; going backwards through the passes, a box needed after
// a full step at distance 3^k along dimension a is the joint reduction of its parts inside the left
// peer's previous window, the own previous window and the right peer's (three disjoint windows that
// tile the new one, Appendix A); after the final step along a (distance d), the whole ring along a
// is the own window [-R, R] plus the offsets above R from the peer at +d (the top of that peer's
// window) and those below -R from the peer at -d, offsets taken in (-side/2, side/2]. Every part is
// again a box the sender holds before the pass; the boxes needed before pass t are the slots of
// state t. On powers of three the window is the only slot (the ordinary schedule).

struct Ivl {
    int lo, hi;  // offsets lo..hi; empty when lo > hi
    bool empty() const { return lo > hi; }
    bool operator==(const Ivl& o) const { return lo == o.lo && hi == o.hi; }
};

Ivl meet(Ivl a, Ivl b) { return Ivl{std::max(a.lo, b.lo), std::min(a.hi, b.hi)}; }

struct SlotBox {
    Ivl iv[kMaxDims];
    bool operator==(const SlotBox& o) const {
        for (int d = 0; d < kMaxDims; ++d)
            if (!(iv[d] == o.iv[d])) return false;
        return true;
    }
};

struct SideSteps {
    int side = 1, f = 0, d = 0;  // full steps, final distance (0: none)
    int steps() const { return side == 1 ? 0 : f + (d ? 1 : 0); }
    int dist(int k) const { return k < f ? ipow3(k) : d; }
    // offsets covered after `taken` steps along this side (Lemma 2 windows, then the whole ring)
    Ivl window(int taken) const {
        if (side == 1) return Ivl{0, 0};
        if (taken > f) {
            const int lo = -((side - 1) / 2);
            return Ivl{lo, lo + side - 1};
        }
        const int R = (ipow3(taken) - 1) / 2;
        return Ivl{-R, R};
    }
};

SideSteps side_steps(int side) {
    SideSteps ss;
    ss.side = side;
    if (side == 1) return ss;
    int pw = 1;
    while (pw * 3 <= side) {
        pw *= 3;
        ss.f += 1;
    }
    ss.d = pw == side ? 0 : (side - pw + 1) / 2;
    return ss;
}

int build_latency_slot_plan(trivance_plan_t* p) {
    const int D = p->D;
    SideSteps ss[kMaxDims];
    p->S = 0;
    for (int d = 0; d < D; ++d) {
        ss[d] = side_steps(p->dims[d]);
        p->S += ss[d].steps();
    }
    const int S = p->S;
    if (S > 40) return TRIVANCE_EUNSUPPORTED;
    std::vector<Pass> passes(S);
    std::vector<trivance::SlotPass> sp(S);
    for (int t = 0; t < S; ++t) {
        passes[t] = Pass{};
        passes[t].phase = TRIVANCE_PHASE_LATENCY;
        passes[t].step = t;
        for (int c = 0; c < kMaxDims; ++c) {
            passes[t].distance[c] = 1;
            for (int dd = 0; dd < kMaxDims; ++dd) passes[t].modulus[c][dd] = 1;
        }
        sp[t] = trivance::SlotPass{};
    }
    p->max_slots = 1;
    for (int c = 0; c < D; ++c) {
        // rotation: the first dimension, cyclically from (c + t) mod D, with steps left
        std::vector<std::vector<int>> taken(S + 1, std::vector<int>(D, 0));
        std::vector<int> act(S), kk(S);
        for (int t = 0; t < S; ++t) {
            int dsel = -1;
            for (int i = 0; i < D && dsel < 0; ++i) {
                const int cand = (c + t + i) % D;
                if (taken[t][cand] < ss[cand].steps()) dsel = cand;
            }
            act[t] = dsel;
            kk[t] = taken[t][dsel];
            taken[t + 1] = taken[t];
            taken[t + 1][dsel] += 1;
            Pass& ps = passes[t];
            ps.dim[c] = dsel;
            ps.dim_step[c] = kk[t];
            ps.distance[c] = ss[dsel].dist(kk[t]);
            for (int dd = 0; dd < D; ++dd) ps.taken[c][dd] = taken[t][dd];
        }
        auto window_box = [&](int t) {
            SlotBox b{};
            for (int dd = 0; dd < kMaxDims; ++dd)
                b.iv[dd] = dd < D ? ss[dd].window(taken[t][dd]) : Ivl{0, 0};
            return b;
        };
        std::vector<SlotBox> need{window_box(S)};
        for (int t = S - 1; t >= 0; --t) {
            const int a = act[t];
            const int dist = ss[a].dist(kk[t]);
            const Ivl prev = ss[a].window(taken[t][a]);
            const Ivl cur = ss[a].window(taken[t + 1][a]);
            const bool final_step = ss[a].d != 0 && kk[t] == ss[a].f;
            std::vector<SlotBox> parts{window_box(t)};
            auto index_of = [&](const SlotBox& b) {
                for (size_t i = 0; i < parts.size(); ++i)
                    if (parts[i] == b) return (int)i;
                parts.push_back(b);
                return (int)parts.size() - 1;
            };
            if ((int)need.size() > trivance::kMaxSlots) return TRIVANCE_EUNSUPPORTED;
            sp[t].nout[c] = (int)need.size();
            for (size_t i = 0; i < need.size(); ++i) {
                const Ivl I = need[i].iv[a];
                if (I.lo < cur.lo || I.hi > cur.hi) return TRIVANCE_EUNSUPPORTED;  // not a window part
                Ivl own, left, right;
                if (final_step) {
                    if (!(I == cur)) return TRIVANCE_EUNSUPPORTED;
                    own = prev;
                    left = Ivl{cur.lo, prev.lo - 1};   // beyond -R: from the peer at -d
                    right = Ivl{prev.hi + 1, cur.hi};  // beyond +R: from the peer at +d
                } else {
                    own = meet(I, prev);
                    left = meet(I, Ivl{cur.lo, prev.lo - 1});
                    right = meet(I, Ivl{prev.hi + 1, cur.hi});
                }
                const Ivl pieces[3] = {own, left, right};
                const int shift[3] = {0, +dist, -dist};  // into the sender's own frame
                int idx[3];
                for (int q = 0; q < 3; ++q) {
                    idx[q] = -1;
                    if (pieces[q].empty()) continue;
                    SlotBox b = need[i];
                    b.iv[a] = Ivl{pieces[q].lo + shift[q], pieces[q].hi + shift[q]};
                    if (b.iv[a].lo < prev.lo || b.iv[a].hi > prev.hi) return TRIVANCE_EUNSUPPORTED;
                    idx[q] = index_of(b);
                }
                sp[t].own[c][i] = (int8_t)idx[0];
                sp[t].left[c][i] = (int8_t)idx[1];
                sp[t].right[c][i] = (int8_t)idx[2];
            }
            if ((int)parts.size() > trivance::kMaxSlots) return TRIVANCE_EUNSUPPORTED;
            sp[t].nin[c] = (int)parts.size();
            p->max_slots = std::max(p->max_slots, (int)parts.size());
            need.swap(parts);
        }
        // before the first pass a rank holds only its own value
        SlotBox start{};
        if (need.size() != 1 || !(need[0] == start)) return TRIVANCE_EUNSUPPORTED;
    }
    p->passes = passes;
    p->slots = sp;
    return TRIVANCE_OK;
}

}  // namespace

namespace trivance {

int placed_position(const trivance_plan_t* p, int c, int block) {
    // reduce-scatter step t (pass t) of collective c works on dimension passes[t].dim[c] and
    // fixes that coordinate's next base-3 digit
    int coord[kMaxDims];
    int rest = block;
    for (int d = 0; d < p->D; ++d) {
        coord[d] = rest % p->dims[d];
        rest /= p->dims[d];
    }
    int pos = 0;
    for (int t = 0; t < p->S; ++t) {
        const int d = p->passes[t].dim[c];
        pos = 3 * pos + coord[d] % 3;
        coord[d] /= 3;
    }
    return pos;
}

void block_bounds(const trivance_plan_t* p, int64_t elems, int c, int block, int64_t* begin,
                  int64_t* end) {
    if (block >= 0 && p->placed) block = placed_position(p, c, block);
    const int64_t G = (elems + kGranule - 1) / kGranule;
    const int64_t g0 = (int64_t)c * G / p->D;
    const int64_t g1 = (int64_t)(c + 1) * G / p->D;
    int64_t b = g0, e = g1;
    if (block >= 0) {
        const int64_t Gc = g1 - g0;
        b = g0 + (int64_t)block * Gc / p->n;
        e = g0 + (int64_t)(block + 1) * Gc / p->n;
    }
    *begin = b * kGranule < elems ? b * kGranule : elems;
    *end = e * kGranule < elems ? e * kGranule : elems;
}

int64_t max_block_granules(const trivance_plan_t* p, int64_t elems) {
    const int64_t G = (elems + kGranule - 1) / kGranule;
    int64_t best = 0;
    for (int c = 0; c < p->D; ++c) {
        const int64_t Gc = (int64_t)(c + 1) * G / p->D - (int64_t)c * G / p->D;
        const int64_t m = (Gc + p->n - 1) / p->n;  // ceil: the largest floor-difference
        if (m > best) best = m;
    }
    return best;
}

}  // namespace trivance

extern "C" {

int trivance_plan(int n, const int* torus_dims, int ndims, int variant, trivance_plan_t** out) {
    return trivance_plan_ex(n, torus_dims, ndims, variant, 0u, out);
}

int trivance_plan_ex(int n, const int* torus_dims, int ndims, int variant, unsigned flags,
                     trivance_plan_t** out) {
    if (!out) return TRIVANCE_EINVAL;
    *out = nullptr;
    if (flags & ~TRIVANCE_PLACE_BY_SCHEDULE) return TRIVANCE_EINVAL;
    if (n < 1 || ndims < 0) return TRIVANCE_EINVAL;
    if (variant < TRIVANCE_LATENCY_OPT || variant > TRIVANCE_BRUCK_REF) return TRIVANCE_EINVAL;
    int dims[kMaxDims] = {};
    int D = ndims;
    if (ndims == 0 || torus_dims == nullptr) {
        D = 1;
        dims[0] = n;
    } else {
        if (ndims > kMaxDims) return TRIVANCE_EUNSUPPORTED;
        long long prod = 1;
        for (int d = 0; d < ndims; ++d) {
            if (torus_dims[d] < 1) return TRIVANCE_EINVAL;
            dims[d] = torus_dims[d];
            prod *= dims[d];
            if (prod > (1LL << 30)) return TRIVANCE_EINVAL;
        }
        if (prod != n) return TRIVANCE_EINVAL;
    }
    bool pow3 = true;
    for (int d = 0; d < D; ++d) pow3 = pow3 && log3_exact(dims[d]) >= 0;
    if ((flags & TRIVANCE_PLACE_BY_SCHEDULE) && (!pow3 || variant != TRIVANCE_BANDWIDTH_OPT))
        return TRIVANCE_EUNSUPPORTED;
    // Sec. 4.4 (sides that are not powers of three): reduction trees (bandwidth-optimal) or slot
    // programs (latency-optimal)
    if (!pow3) {
        if (variant == TRIVANCE_BRUCK_REF || D > trivance::kMaxTreeDims) return TRIVANCE_EUNSUPPORTED;
        for (int d = 0; d < D; ++d)
            if (dims[d] > trivance::kMaxTreeSide) return TRIVANCE_EUNSUPPORTED;
    }
    if (variant == TRIVANCE_BRUCK_REF && D != 1) return TRIVANCE_EUNSUPPORTED;

    trivance_plan_t* p = new (std::nothrow) trivance_plan_t;
    if (!p) return TRIVANCE_ENOMEM;
    p->n = n;
    p->D = D;
    p->variant = variant;
    if (!pow3) {
        int stride1 = 1;
        for (int d = 0; d < D; ++d) {
            p->dims[d] = dims[d];
            p->strides[d] = stride1;
            stride1 *= dims[d];
        }
        int rc;
        try {
            rc = variant == TRIVANCE_BANDWIDTH_OPT ? build_tree_plan(p) : build_latency_slot_plan(p);
        } catch (const std::bad_alloc&) {
            rc = TRIVANCE_ENOMEM;
        }
        if (rc != TRIVANCE_OK) {
            delete p;
            return rc;
        }
        *out = p;
        return TRIVANCE_OK;
    }
    int stride = 1;
    int steps_per_dim[kMaxDims] = {};
    for (int d = 0; d < D; ++d) {
        p->dims[d] = dims[d];
        p->strides[d] = stride;
        stride *= dims[d];
        steps_per_dim[d] = log3_exact(dims[d]);
        p->S += steps_per_dim[d];
    }
    if (p->S > 64) {
        delete p;
        return TRIVANCE_EUNSUPPORTED;
    }
    Rotation* rot = new (std::nothrow) Rotation;
    if (!rot) {
        delete p;
        return TRIVANCE_ENOMEM;
    }
    fill_rotation(p, steps_per_dim, rot);
    try {
        if (variant == TRIVANCE_BANDWIDTH_OPT) {
            for (int t = 0; t < p->S; ++t)
                p->passes.push_back(make_pass(p, *rot, TRIVANCE_PHASE_REDUCE_SCATTER, t));
            for (int t = p->S - 1; t >= 0; --t)
                p->passes.push_back(make_pass(p, *rot, TRIVANCE_PHASE_ALLGATHER, t));
        } else {
            for (int t = 0; t < p->S; ++t)
                p->passes.push_back(make_pass(p, *rot, TRIVANCE_PHASE_LATENCY, t));
        }
    } catch (const std::bad_alloc&) {
        delete rot;
        delete p;
        return TRIVANCE_ENOMEM;
    }
    delete rot;
    p->placed = (flags & TRIVANCE_PLACE_BY_SCHEDULE) != 0;
    *out = p;
    return TRIVANCE_OK;
}

void trivance_plan_destroy(trivance_plan_t* plan) { delete plan; }

int trivance_plan_num_steps(const trivance_plan_t* plan) {
    return plan ? plan->S : TRIVANCE_EINVAL;
}

int trivance_plan_num_passes(const trivance_plan_t* plan) {
    return plan ? (int)plan->passes.size() : TRIVANCE_EINVAL;
}

int trivance_plan_step(const trivance_plan_t* plan, int pass, int collective, int* phase,
                       int* dim, int* distance) {
    if (!plan || pass < 0 || pass >= (int)plan->passes.size() || collective < 0 ||
        collective >= plan->D)
        return TRIVANCE_EINVAL;
    const Pass& ps = plan->passes[pass];
    if (phase) *phase = ps.phase;
    if (dim) *dim = ps.dim[collective];
    if (distance) *distance = ps.distance[collective];
    return TRIVANCE_OK;
}

int trivance_plan_step_index(const trivance_plan_t* plan, int pass) {
    if (!plan || pass < 0 || pass >= (int)plan->passes.size()) return TRIVANCE_EINVAL;
    return plan->passes[pass].step;
}

int trivance_plan_with_dispatch_limit(const trivance_plan_t* plan, int64_t work_items,
                                      trivance_plan_t** out) {
    if (!out) return TRIVANCE_EINVAL;
    *out = nullptr;
    if (!plan || work_items < 1024 || work_items > trivance::kMaxDispatchItems)
        return TRIVANCE_EINVAL;
    trivance_plan_t* p = nullptr;
    try {
        p = new trivance_plan_t(*plan);
    } catch (const std::bad_alloc&) {
        return TRIVANCE_ENOMEM;
    }
    p->dispatch_items = work_items;
    *out = p;
    return TRIVANCE_OK;
}

int trivance_block_range(const trivance_plan_t* plan, int64_t elems, int collective, int block,
                         int64_t* begin, int64_t* end) {
    if (!plan || !begin || !end || elems < 0 || collective < 0 || collective >= plan->D ||
        block < -1 || block >= plan->n)
        return TRIVANCE_EINVAL;
    trivance::block_bounds(plan, elems, collective, block, begin, end);
    return TRIVANCE_OK;
}

int64_t trivance_pass_bytes(const trivance_plan_t* plan, int64_t elems, int dtype, int pass) {
    if (!plan || elems < 0 || pass < 0 || pass >= (int)plan->passes.size()) return TRIVANCE_EINVAL;
    if (dtype != TRIVANCE_F32 && dtype != TRIVANCE_I32) return TRIVANCE_EINVAL;
    const int64_t w = 4;
    const Pass& ps = plan->passes[pass];
    const int64_t n = plan->n;
    if (ps.phase == TRIVANCE_PHASE_LATENCY && !plan->slots.empty()) {
        // every rank reads each slot it holds before the pass once and writes each slot it holds
        // after it once, over its collective's segment
        const trivance::SlotPass& sp = plan->slots[pass];
        int64_t acc = 0;
        for (int c = 0; c < plan->D; ++c) {
            int64_t b, e;
            trivance::block_bounds(plan, elems, c, -1, &b, &e);
            acc += (int64_t)(sp.nin[c] + sp.nout[c]) * n * (e - b);
        }
        return acc * w;
    }
    if (ps.phase == TRIVANCE_PHASE_LATENCY) return 2 * n * elems * w;
    if (plan->tree) {
        // Collective c's pass touches, for every block j of its segment, the ranks j + o with o
        // a receiver offset in the active dimension and an offset not yet forwarded in every
        // other; all blocks of a segment together cover the segment. A receiver reads its own
        // partial and each sending child and writes once (reduce-scatter), or reads once and
        // writes to each child (all-gather).
        int64_t acc = 0;
        for (int c = 0; c < plan->D; ++c) {
            const int a = ps.dim[c];
            int64_t per = 0;
            for (uint32_t r : plan->trees[a].recv[ps.dim_step[c]]) {
                const int64_t kids = ((r & trivance::kFromLeft) ? 1 : 0) + ((r & trivance::kFromRight) ? 1 : 0);
                per += ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER ? 2 + kids : 1 + kids;
            }
            for (int d = 0; d < plan->D; ++d)
                if (d != a) per *= (int64_t)plan->trees[d].alive[ps.taken[c][d]].size();
            int64_t b, e;
            trivance::block_bounds(plan, elems, c, -1, &b, &e);
            acc += per * (e - b);
        }
        return acc * w;
    }
    // Every (centre rank r, kept block j) pair of the pass touches block j in three rows:
    // reduce-scatter reads own/left/right and writes own (4 accesses); all-gather reads the
    // centre and writes both peers (3 accesses). Each block index j has exactly n / 3^(t+1)
    // centres, and the blocks of all segments add up to the whole vector, so the pairs cover
    // kept_per_rank * elems elements.
    const int64_t covered = ps.kept_per_rank * elems;
    const int64_t accesses = ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER ? 4 : 3;
    return accesses * covered * w;
}

int64_t trivance_algorithmic_bytes(const trivance_plan_t* plan, int64_t elems, int dtype) {
    if (!plan) return TRIVANCE_EINVAL;
    int64_t total = 0;
    for (int p = 0; p < (int)plan->passes.size(); ++p) {
        const int64_t b = trivance_pass_bytes(plan, elems, dtype, p);
        if (b < 0) return b;
        total += b;
    }
    return total;
}

const char* trivance_strerror(int status) {
    switch (status) {
        case TRIVANCE_OK: return "success";
        case TRIVANCE_EINVAL: return "invalid argument";
        case TRIVANCE_EUNSUPPORTED: return "unsupported configuration";
        case TRIVANCE_EHIP: return "HIP runtime error";
        case TRIVANCE_ENOMEM: return "out of host memory";
        case TRIVANCE_ESIZE: return "output buffer too small";
        case TRIVANCE_ESCRATCH: return "request exceeds the fixed device scratch";
        default: return "unknown status";
    }
}

}  // extern "C"
