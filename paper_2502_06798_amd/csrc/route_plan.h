// Route-Plan (Eq. 1): an optimal integer plan X[i][j] = queries of optimal
// level i served at level j, given the batch's demand H per level, the
// capacity F per level and the skipped steps K (K_0 = 0 < K_1 < .. < K_L).
//
// Serving level i at j > i degrades it by K_j - K_i, serving it at j <= i
// costs nothing, and an optimum serves min(sum H, sum F) queries.  Moving a
// query from i up to j crosses the boundaries i|i+1 .. j-1|j once each and
// costs the sum of K_{m+1} - K_m over them, so a plan's degradation is
//   sum_m (K_{m+1} - K_m) * (queries crossing boundary m|m+1 upwards),
// and no plan crosses boundary m upwards fewer than
//   E_m = sum_{i<=m} H_i - sum_{i<=m} F_i
// times.  The plan below meets every bound at once, so it is optimal:
//   1. excess demand (sum H - sum F, if positive) is left unserved from the
//      lowest levels up (this lowers every E_m the most);
//   2. every level serves its own queries first: y_i = min(H_i, F_i), leaving
//      demand r_i or room c_i (never both);
//   3. the net flow across boundary m is n_m = max(E_m, -A_m) upwards, with
//      E_m over the leftovers r - c and A_m = sum_{i>m} r_i (a negative n_m
//      sends queries down into free room, which costs nothing);
//   4. the queries that move up (down) are matched to the room they fill in
//      first-in-first-out order along the upward (downward) sweep, so the
//      k-th query to leave its level fills the k-th place; X[i][j] is the
//      overlap of i's interval of departures with j's interval of arrivals.
// Every step is per level (steps 1-3, prefix sums over levels) or per plan
// entry (step 4), so the same functions run as host loops and as one thread
// per level / per entry on the device.
#pragma once
#include <stdint.h>

#include "../../include/apc.h"

namespace apc {

#if defined(__HIPCC__)
#define APC_HD __host__ __device__
#else
#define APC_HD
#endif

struct PlanWork {
    int32_t y[APC_MAX_LEVELS + 1];          // served at the own level
    int32_t r[APC_MAX_LEVELS + 1];          // demand left after that
    int32_t c[APC_MAX_LEVELS + 1];          // room left after that
    int32_t n[APC_MAX_LEVELS + 1];          // net upward flow across boundary m|m+1 (n[L] = 0)
    int32_t up0[APC_MAX_LEVELS + 1], up1[APC_MAX_LEVELS + 1];   // departures [up0, up1) upwards
    int32_t ua0[APC_MAX_LEVELS + 1], ua1[APC_MAX_LEVELS + 1];   // arrivals from below
    int32_t dn0[APC_MAX_LEVELS + 1], dn1[APC_MAX_LEVELS + 1];   // departures downwards
    int32_t da0[APC_MAX_LEVELS + 1], da1[APC_MAX_LEVELS + 1];   // arrivals from above
};

// Step 1 and 2 for level m.
APC_HD inline void plan_level_own(int L, const int32_t* H, const int32_t* F, int m, PlanWork& w)
{
    int64_t sh = 0, sf = 0, below = 0;
    for (int i = 0; i <= L; ++i) {
        sh += H[i];
        sf += F[i];
        if (i < m) below += H[i];
    }
    const int64_t unserved = sh > sf ? sh - sf : 0;
    int64_t drop = unserved - below;
    drop = drop < 0 ? 0 : (drop > H[m] ? H[m] : drop);
    const int32_t h = H[m] - (int32_t)drop;
    const int32_t y = h < F[m] ? h : F[m];
    w.y[m] = y;
    w.r[m] = h - y;
    w.c[m] = F[m] - y;
}

// Step 3 for boundary m|m+1 (m < L); needs r and c of every level.
APC_HD inline void plan_level_flow(int L, int m, PlanWork& w)
{
    int64_t e = 0, a = 0;
    for (int i = 0; i <= L; ++i) {
        if (i <= m) e += (int64_t)w.r[i] - w.c[i];
        else a += w.r[i];
    }
    w.n[m] = (int32_t)(e > -a ? e : -a);
}

// Departure and arrival counts of level m; needs n of every boundary.
APC_HD inline void plan_level_moves(int m, const PlanWork& w, int32_t& up, int32_t& ua, int32_t& dn, int32_t& da)
{
    const int32_t lo = m > 0 ? w.n[m - 1] : 0, hi = w.n[m];
    const int32_t uin = lo > 0 ? lo : 0, uout = hi > 0 ? hi : 0;     // up from below / up to above
    const int32_t din = hi < 0 ? -hi : 0, dout = lo < 0 ? -lo : 0;   // down from above / down to below
    if (w.r[m] > 0) {                       // demand level: queries leave, none stay
        up = uout - uin;
        dn = dout - din;
        ua = da = 0;
    } else {                                // room (or idle) level: queries stop here
        up = dn = 0;
        ua = uin - uout;
        da = din - dout;
    }
}

// Step 4 intervals of level m (prefix sums of the counts in sweep order).
APC_HD inline void plan_level_intervals(int L, int m, PlanWork& w)
{
    int32_t pu = 0, pa = 0, pd = 0, pda = 0;
    int32_t up = 0, ua = 0, dn = 0, da = 0;
    for (int i = 0; i < m; ++i) {           // upward sweep: levels below m go first
        plan_level_moves(i, w, up, ua, dn, da);
        pu += up;
        pa += ua;
    }
    for (int i = L; i > m; --i) {           // downward sweep: levels above m go first
        plan_level_moves(i, w, up, ua, dn, da);
        pd += dn;
        pda += da;
    }
    plan_level_moves(m, w, up, ua, dn, da);
    w.up0[m] = pu;  w.up1[m] = pu + up;
    w.ua0[m] = pa;  w.ua1[m] = pa + ua;
    w.dn0[m] = pd;  w.dn1[m] = pd + dn;
    w.da0[m] = pda; w.da1[m] = pda + da;
}

APC_HD inline int32_t plan_overlap(int32_t a0, int32_t a1, int32_t b0, int32_t b1)
{
    const int32_t lo = a0 > b0 ? a0 : b0, hi = a1 < b1 ? a1 : b1;
    return hi > lo ? hi - lo : 0;
}

// Step 4: the plan entry X[i][j].
APC_HD inline int32_t plan_entry(int i, int j, const PlanWork& w)
{
    if (i == j) return w.y[i];
    if (j > i) return plan_overlap(w.up0[i], w.up1[i], w.ua0[j], w.ua1[j]);
    return plan_overlap(w.dn0[i], w.dn1[i], w.da0[j], w.da1[j]);
}

// Host: the whole plan, X row-major (L+1) x (L+1).
inline void plan_route_host(int L, const int32_t* H, const int32_t* F, int32_t* X)
{
    PlanWork w;
    for (int m = 0; m <= L; ++m) plan_level_own(L, H, F, m, w);
    for (int m = 0; m < L; ++m) plan_level_flow(L, m, w);
    w.n[L] = 0;
    for (int m = 0; m <= L; ++m) plan_level_intervals(L, m, w);
    for (int i = 0; i <= L; ++i)
        for (int j = 0; j <= L; ++j) X[i * (L + 1) + j] = plan_entry(i, j, w);
}

}  // namespace apc
