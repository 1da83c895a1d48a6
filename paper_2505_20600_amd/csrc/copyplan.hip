// Cache-load plan of one request (block-wise loading, Sec. 4.2 and Fig. 8:
// a cached block loads the cached activations of the unmasked image tokens
// only). Host code, no device work.
//
// A copy command costs the copy engine a fixed time on top of its bytes, so
// one copy per unmasked run would crawl at the masks' blob edges, and merging
// runs across masked gaps moves masked rows for nothing. A strided 2-D copy
// moves equally long runs spaced one grid row apart as ONE command at the
// link's full rate (measured on MI355X from pinned host memory: 64 rows of
// 96 KiB at 52.9 GB/s in one 2-D copy, 8.6 GB/s as 64 copies). On the token
// grid, a masked rectangle `hole` spanning grid rows [y0, y1) is skipped by
// such copies: the runs between the holes of each grid row repeat row after
// row. The planner therefore
//   1. chains the masked intervals of consecutive grid rows into tracks
//      (one interval per row, linked to an overlapping interval above),
//   2. splits each track into bands of rows by dynamic programming; a band
//      either skips the rectangle common to its rows (one more command,
//      the band's other masked cells still copied) or copies all its masked
//      cells, whichever the cost model prices lower,
//   3. covers everything outside the chosen holes with maximal runs in token
//      order, a run that repeats the run one grid row earlier joining that
//      run's strided copy,
//   4. drops, one at a time, holes whose removal lowers the modelled cost
//      (band boundaries add commands the band-wise model does not see; bands
//      and this pass are bounded so that the host time stays linear in the
//      tokens),
//   5. keeps the plan only if it is cheaper than plain runs merged across
//      gaps shorter than one command's cost.
// Cost model: every command costs `C` rows of link time, plus one row per row
// moved.
#include <algorithm>
#include <unordered_map>
#include <vector>

#include "step_internal.h"

namespace ms {
namespace {

struct Iv {
    int a, e;   // masked columns [a, e) of one grid row
};

struct Hole {
    int x0, x1, y0, y1;   // masked columns [x0, x1) of grid rows [y0, y1)
};

// Bounds on the planner's host time for tall grids and busy masks: bands of
// at most kMaxBandRows rows (the band search is linear in the track length
// times this), and the hole-dropping pass (each trial rebuilds the plan) only
// while holes x tokens stays below kDropWork.
constexpr int kMaxBandRows = 256;
constexpr int64_t kDropWork = int64_t(1) << 26;

double plan_cost(const std::vector<CopyRect>& p, double C) {
    double c = 0.0;
    for (const CopyRect& r : p) c += C + (double)r.w * r.h;
    return c;
}

// Plain runs of unmasked rows, merged across masked gaps of at most `gap` rows.
void merged_runs(const uint8_t* m, int N, int gap, std::vector<CopyRect>& out) {
    out.clear();
    int n = 0;
    while (n < N) {
        while (n < N && m[n]) ++n;
        if (n >= N) break;
        const int n0 = n;
        while (n < N && !m[n]) ++n;
        if (!out.empty() && n0 - (out.back().n0 + out.back().w) <= gap)
            out.back().w = n - out.back().n0;
        else
            out.push_back(CopyRect{n0, n - n0, 1});
    }
}

// Copies of every row outside `holes` (step 3): `keep` is scratch.
void copies_outside(const std::vector<Hole>& holes, const std::vector<char>& live, int H, int P,
                    std::vector<uint8_t>& keep, std::vector<CopyRect>& out) {
    const int N = H * P;
    keep.assign((size_t)N, 1);
    for (size_t i = 0; i < holes.size(); ++i) {
        if (!live[i]) continue;
        const Hole& h = holes[i];
        for (int y = h.y0; y < h.y1; ++y) std::fill(keep.begin() + (size_t)y * P + h.x0, keep.begin() + (size_t)y * P + h.x1, 0);
    }
    out.clear();
    std::unordered_map<int, int> next;   // start row a strided copy expects next -> its index
    int n = 0;
    while (n < N) {
        while (n < N && !keep[n]) ++n;
        if (n >= N) break;
        const int a = n;
        while (n < N && keep[n]) ++n;
        const int w = n - a;
        auto it = next.find(a);
        if (it != next.end() && out[it->second].w == w && w < P) {
            const int k = it->second;
            next.erase(it);
            ++out[k].h;
            next[a + P] = k;
        } else {
            if (it != next.end()) next.erase(it);
            out.push_back(CopyRect{a, w, 1});
            if (w < P) next[a + P] = (int)out.size() - 1;
        }
    }
}

// Steps 1 and 2: candidate holes of one request's mask [H][P].
void band_holes(const uint8_t* m, int H, int P, double C, std::vector<Hole>& holes) {
    holes.clear();
    struct Track {
        int y0;
        std::vector<Iv> iv;
    };
    std::vector<Track> tracks;
    std::vector<std::pair<Iv, int>> prev, cur;   // intervals of the row above / this row, with their track
    std::vector<int> used_in_row;                // last row each track took an interval in
    for (int y = 0; y < H; ++y) {
        cur.clear();
        const uint8_t* r = m + (size_t)y * P;
        size_t p = 0;
        int x = 0;
        while (x < P) {
            while (x < P && !r[x]) ++x;
            if (x >= P) break;
            const int a = x;
            while (x < P && r[x]) ++x;
            const Iv iv{a, x};
            // the first interval above that overlaps this one and whose track
            // has no interval in this row yet (both rows are sorted: `p` only
            // moves forward)
            while (p < prev.size() && prev[p].first.e <= iv.a) ++p;
            int t = -1;
            for (size_t q = p; q < prev.size() && prev[q].first.a < iv.e; ++q)
                if (used_in_row[prev[q].second] != y) {
                    t = prev[q].second;
                    break;
                }
            if (t < 0) {
                t = (int)tracks.size();
                tracks.push_back(Track{y, {}});
                used_in_row.push_back(-1);
            }
            used_in_row[t] = y;
            tracks[t].iv.push_back(iv);
            cur.emplace_back(iv, t);
        }
        prev.swap(cur);
    }
    std::vector<double> dp;
    std::vector<int> from;
    std::vector<Hole> pick;
    for (const Track& tr : tracks) {
        const int n = (int)tr.iv.size();
        dp.assign(n + 1, 0.0);
        from.assign(n + 1, 0);
        pick.assign(n + 1, Hole{0, 0, 0, 0});
        for (int i = 1; i <= n; ++i) {
            // the band's last row alone, its masked cells copied
            dp[i] = dp[i - 1] + (tr.iv[i - 1].e - tr.iv[i - 1].a);
            from[i] = i - 1;
            pick[i] = Hole{0, 0, 0, 0};
            int lo = 0, hi = P;
            double masked = 0.0;
            for (int j = i - 1; j >= std::max(0, i - kMaxBandRows); --j) {
                lo = std::max(lo, tr.iv[j].a);
                hi = std::min(hi, tr.iv[j].e);
                if (hi <= lo) break;   // no common rectangle for this band or any longer one
                masked += tr.iv[j].e - tr.iv[j].a;
                const double c = dp[j] + C + masked - (double)(hi - lo) * (i - j);
                if (c < dp[i]) {
                    dp[i] = c;
                    from[i] = j;
                    pick[i] = Hole{lo, hi, tr.y0 + j, tr.y0 + i};
                }
            }
        }
        for (int i = n; i > 0; i = from[i])
            if (pick[i].x1 > pick[i].x0) holes.push_back(pick[i]);
    }
}

}  // namespace

void plan_copies(const uint8_t* m, int H, int P, double C, bool strided, std::vector<CopyRect>& out) {
    const int N = H * P;
    // step 5's baseline: gaps shorter than one command's cost merge
    std::vector<CopyRect> runs;
    merged_runs(m, N, (int)std::min(C, (double)N), runs);
    if (!strided) {
        out.swap(runs);
        return;
    }
    const double runs_cost = plan_cost(runs, C);

    std::vector<Hole> holes;
    band_holes(m, H, P, C, holes);
    std::vector<char> live(holes.size(), 1);
    std::vector<uint8_t> keep;
    std::vector<CopyRect> plan, trial;
    copies_outside(holes, live, H, P, keep, plan);
    double best = plan_cost(plan, C);
    // step 4: smallest holes first
    std::vector<int> order(holes.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
        return (int64_t)(holes[a].x1 - holes[a].x0) * (holes[a].y1 - holes[a].y0) <
               (int64_t)(holes[b].x1 - holes[b].x0) * (holes[b].y1 - holes[b].y0);
    });
    if ((int64_t)holes.size() * N > kDropWork) order.clear();
    for (int i : order) {
        live[i] = 0;
        copies_outside(holes, live, H, P, keep, trial);
        const double c = plan_cost(trial, C);
        if (c < best) {
            best = c;
            plan.swap(trial);
        } else {
            live[i] = 1;
        }
    }
    if (best < runs_cost) out.swap(plan);
    else out.swap(runs);
}

}  // namespace ms
