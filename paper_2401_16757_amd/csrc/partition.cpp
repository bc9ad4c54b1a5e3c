// partition.cpp -- delay model of a swapped run and the search for the slab
// partition that minimises it.
//
// Sec. 5 gives each block three delays: an input delay (swap-in, linear in
// the block's bytes, plus assembly, linear in its parameter depth), an
// execution delay (linear in its FLOPs) and an output delay (swap-out).
// Sec. 6 then picks the number of blocks and the partition points that
// minimise the total time under the pair constraint (Eq. 3), from delays
// predicted by those linear models.  Here the same three delays are modelled
// for this engine: one DMA per slab (t_in = alpha * bytes + beta; binding by
// pointer costs the device nothing), per-layer execution times (measured, or
// gamma * FLOPs + kappa), and no swap-out work (a slab's range is reused once
// its compute has finished).  Instead of the recurrence over residual
// overlaps, the time of a partition is read off a replay of the engine's own
// schedule: the DMA queue in slab order, each swap-in waiting for the compute
// of the slab whose range it overwrites (its `wait` slab, or one inference
// earlier its `wrap` slab), each slab's compute waiting for its swap-in and
// for the previous slab.  The search over partitions replaces the paper's
// precomputed lookup table: every candidate count n around ceil(2 s / b) is
// started from equal-byte cuts and improved by moving single cut points.
#include <math.h>

#include <algorithm>
#include <limits>

#include "engine.h"

namespace sn {

double layer_flops(const Layer &L) {
    const sn_layer &d = L.d;
    switch (d.op) {
    case SN_OP_CONV2D:
        return 2.0 * L.out_h * L.out_w * d.c_out * (double)d.c_in * d.k * d.k;
    case SN_OP_LINEAR:   // per token for token networks
        return 2.0 * d.c_out * L.rows_per_unit * (double)d.c_in;
    default:
        return 0.0;
    }
}

static double layer_seconds(const std::vector<Layer> &layers, int li, const CostModel &m) {
    if (li < (int)m.layer_ex.size() && m.layer_ex[li] >= 0) return m.layer_ex[li];
    return m.gamma * layer_flops(layers[li]) + m.kappa;
}

// A slice of a layer keeps the fixed part (kappa) of the layer's time whole
// and a share of the rest proportional to its output units.
static double piece_seconds(const std::vector<Layer> &layers, const Piece &p, const CostModel &m) {
    const Layer &L = layers[p.layer];
    const double t = layer_seconds(layers, p.layer, m);
    if (!L.units || p.u1 - p.u0 >= L.units) return t;
    const double fixed = std::min(m.kappa, t);
    return fixed + (t - fixed) * (double)(p.u1 - p.u0) / (double)L.units;
}

PlanTimes simulate_plan(const std::vector<Layer> &layers, const PlanResult &p, const CostModel &m) {
    const int n = (int)p.slabs.size();
    std::vector<double> ex(n, m.slab_ex);
    for (int i = 0; i < n; ++i)
        for (int pi : p.slabs[i].pieces) ex[i] += piece_seconds(layers, p.pieces[pi], m);
    PlanTimes out;
    if (p.resident) {
        for (double t : ex) out.latency += t;
        out.period = out.latency;
        return out;
    }
    // four inferences back to back from an idle start; the period is the
    // mean spacing of the last three completions
    constexpr int K = 4;
    std::vector<double> cur(n, 0.0), prev(n, 0.0);
    double dma_free = 0, comp_free = 0, end[K];
    for (int k = 0; k < K; ++k) {
        for (int i = 0; i < n; ++i) {
            const Slab &s = p.slabs[i];
            double ready = 0;
            if (s.wait >= 0) ready = cur[s.wait] + m.gate;
            else if (s.wrap >= 0 && k > 0) ready = prev[s.wrap] + m.gate;
            // (a slab without weights issues no DMA)
            const double dma_end =
                std::max(dma_free, ready) + (s.bytes ? m.alpha * (double)s.bytes + m.beta : 0.0);
            dma_free = dma_end;
            cur[i] = std::max(comp_free, dma_end + m.wake) + ex[i];
            comp_free = cur[i];
        }
        end[k] = comp_free;
        prev = cur;
    }
    out.latency = end[0];
    out.period = (end[K - 1] - end[1]) / (K - 2);
    return out;
}

namespace {
bool better(const PlanTimes &a, const PlanTimes &b) {
    const double tol = 1e-9 * std::max(a.period, b.period);
    if (a.period < b.period - tol) return true;
    if (a.period > b.period + tol) return false;
    return a.latency < b.latency - 1e-9 * std::max(a.latency, b.latency);
}
}  // namespace

int search_partition(const std::vector<Layer> &layers, int64_t B, int64_t arena_budget,
                     int64_t max_slab, const CostModel &m, const std::vector<std::vector<SlabSpec>> &seeds,
                     std::vector<SlabSpec> &best, std::string &err) {
    const int64_t cap = max_slab > 0 ? std::min(B, max_slab) : B;
    // Atoms: whole layers, with layers above 1/16 of the budget cut into
    // equal runs of output units (the finest cut points the search uses).
    const int64_t grain = std::max<int64_t>(kAlign, B / 16);
    std::vector<PieceSpec> atoms;
    std::vector<int64_t> prefix(1, 0);
    for (int li = 0; li < (int)layers.size(); ++li) {
        const Layer &L = layers[li];
        const int64_t u1 = L.units ? L.units : 0;
        const int64_t bytes = spec_bytes(layers, SlabSpec{PieceSpec{li, 0, u1}});
        const bool splittable = L.units >= 2 && L.d.op != SN_OP_EMBED;
        const int64_t parts = splittable ? std::min<int64_t>(u1, std::max<int64_t>(1, (bytes + grain - 1) / grain)) : 1;
        for (int64_t k = 0; k < parts; ++k) {
            PieceSpec a{li, u1 * k / parts, u1 * (k + 1) / parts};
            atoms.push_back(a);
            prefix.push_back(prefix.back() + spec_bytes(layers, SlabSpec{a}));
        }
    }
    const int A = (int)atoms.size();
    const int64_t total = prefix.back();

    std::vector<SlabSpec> specs;
    auto build = [&](const std::vector<int> &cuts) {
        specs.clear();
        int a = 0;
        for (size_t c = 0; c <= cuts.size(); ++c) {
            const int b = c < cuts.size() ? cuts[c] : A;
            SlabSpec ss;
            for (int t = a; t < b; ++t) {
                const PieceSpec &x = atoms[t];
                if (!ss.empty() && ss.back().layer == x.layer && ss.back().u1 == x.u0) ss.back().u1 = x.u1;
                else ss.push_back(x);
            }
            specs.push_back(ss);
            a = b;
        }
    };
    PlanResult pr;
    std::string perr;
    auto eval_specs = [&](const std::vector<SlabSpec> &ss, PlanTimes &t) {
        std::vector<int64_t> sz(ss.size());
        for (size_t i = 0; i < ss.size(); ++i) {
            sz[i] = spec_bytes(layers, ss[i]);
            if (sz[i] > cap) return false;
            if (i > 0 && sz[i - 1] + sz[i] > B) return false;
        }
        layout_slabs(layers, ss, pr);
        if (place_slabs(pr, arena_budget, perr)) return false;
        t = simulate_plan(layers, pr, m);
        return true;
    };
    auto eval_cuts = [&](const std::vector<int> &cuts, PlanTimes &t) {
        build(cuts);
        return eval_specs(specs, t);
    };

    bool have = false;
    PlanTimes best_t;
    for (const std::vector<SlabSpec> &s : seeds) {
        PlanTimes t;
        if (eval_specs(s, t) && (!have || better(t, best_t))) {
            best = s;
            best_t = t;
            have = true;
        }
    }
    const int n_lo = (int)std::max<int64_t>(1, (2 * total + B - 1) / std::max<int64_t>(B, 1) - 1);
    const int n_hi = std::min(A, n_lo + 12);
    // time of each atom under the model (its share of its layer)
    std::vector<double> tprefix(1, 0.0);
    for (const PieceSpec &a : atoms) {
        Piece pc;
        pc.layer = a.layer;
        pc.u0 = a.u0;
        pc.u1 = a.u1;
        tprefix.push_back(tprefix.back() + piece_seconds(layers, pc, m));
    }
    // n - 1 cuts splitting the running sum `pre` into equal parts
    auto equal_cuts = [&](const auto &pre, int n, std::vector<int> &cuts) {
        cuts.clear();
        const double tot = (double)pre.back();
        for (int k = 1; k < n; ++k) {
            const double target = tot * k / n;
            int j = 1;
            while (j < A && (double)pre[j] < target) ++j;
            if (j > 1 && target - (double)pre[j - 1] < (double)pre[j] - target) --j;
            j = std::max(j, cuts.empty() ? 1 : cuts.back() + 1);
            if (j > A - (n - k)) return false;
            cuts.push_back(j);
        }
        return true;
    };
    // coordinate descent: each cut in turn to its best position within a
    // window, then adjacent pairs of cuts shifted together
    auto improve = [&](std::vector<int> &cuts, PlanTimes &cur, bool &ok) {
        const int nc = (int)cuts.size();
        for (int pass = 0; pass < 24; ++pass) {
            bool moved = false;
            for (int j = 0; j < nc; ++j) {
                const int lo = std::max(j == 0 ? 1 : cuts[j - 1] + 1, cuts[j] - 24);
                const int hi = std::min(j == nc - 1 ? A - 1 : cuts[j + 1] - 1, cuts[j] + 24);
                const int orig = cuts[j];
                int pick = orig;
                for (int c = lo; c <= hi; ++c) {
                    if (c == orig) continue;
                    cuts[j] = c;
                    PlanTimes t;
                    if (eval_cuts(cuts, t) && (!ok || better(t, cur))) {
                        pick = c;
                        cur = t;
                        ok = true;
                    }
                }
                cuts[j] = pick;
                moved |= pick != orig;
            }
            for (int j = 0; j + 1 < nc; ++j) {
                for (int d : {-2, -1, 1, 2}) {
                    const int a = cuts[j] + d, b = cuts[j + 1] + d;
                    if (a < (j == 0 ? 1 : cuts[j - 1] + 1) || b > (j + 1 == nc - 1 ? A - 1 : cuts[j + 2] - 1))
                        continue;
                    std::vector<int> trial = cuts;
                    trial[j] = a;
                    trial[j + 1] = b;
                    PlanTimes t;
                    if (eval_cuts(trial, t) && (!ok || better(t, cur))) {
                        cuts = trial;
                        cur = t;
                        ok = true;
                        moved = true;
                    }
                }
            }
            if (!moved) break;
        }
    };
    for (int n = n_lo; n <= n_hi; ++n) {
        // two starts per slab count: equal bytes and equal execution time
        for (int start = 0; start < 2; ++start) {
            std::vector<int> cuts;
            if (!(start == 0 ? equal_cuts(prefix, n, cuts) : equal_cuts(tprefix, n, cuts))) continue;
            PlanTimes cur;
            bool ok = eval_cuts(cuts, cur);
            improve(cuts, cur, ok);
            if (ok && (!have || better(cur, best_t))) {
                build(cuts);
                best = specs;
                best_t = cur;
                have = true;
            }
        }
    }
    if (!have) {
        err = "infeasible: no partition satisfies the pair constraint";
        return SN_E_INFEASIBLE;
    }
    return SN_OK;
}

}  // namespace sn
