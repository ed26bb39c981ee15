// Partial brownout (Sec. 2.2: zero, partial and full brownout; Sec. 5,
// baselines: threshold 1.0 keeps every original expert, 0 substitutes every
// call; Sec. 4.3, closing paragraph: the gate still picks the experts and only
// the calls of eligible cold experts go to their united expert through the
// saved map; Sec. 4.5: the serving controller moves the threshold).
//
// Host only. The hot set is the longest run of experts, taken in order of
// decreasing calibration frequency (ties: lower index first), whose
// cumulative normalised frequency stays at or below theta (plus a 1e-9 slack,
// so theta = 1 keeps every expert whatever the rounding of the sum). The
// layer then runs over S segments: the hot experts in ascending index with
// their own FFN, then the united experts that still have a cold member in
// ascending group index. The segment map e2s replaces e2g in every call.
#include <math.h>

#include <algorithm>
#include <vector>

#include "bmoe_common.h"

extern "C" bmoe_status bmoe_partial_segment_map(const double* freq, const int32_t* e2g, int32_t E, int32_t G,
                                                double theta, int32_t* e2s, int32_t* seg_kind, int32_t* seg_id,
                                                int32_t* n_seg) {
    if (!freq || !e2g || !e2s || !seg_kind || !seg_id || !n_seg) return BMOE_ERR_NULL;
    if (E < 1 || E > BMOE_MAX_EXPERTS || G < 1 || G > E) return BMOE_ERR_SHAPE;
    if (!(theta >= 0.0 && theta <= 1.0)) return BMOE_ERR_SHAPE;
    double tot = 0.0;
    for (int e = 0; e < E; ++e) {
        if (!(freq[e] >= 0.0) || !isfinite(freq[e])) return BMOE_ERR_SHAPE;
        if (e2g[e] < 0 || e2g[e] >= G) return BMOE_ERR_MAP;
        tot += freq[e];
    }
    if (!(tot > 0.0) || !isfinite(tot)) return BMOE_ERR_SHAPE;

    std::vector<int> order(E);
    for (int e = 0; e < E; ++e) order[e] = e;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
        return freq[a] != freq[b] ? freq[a] > freq[b] : a < b;
    });
    std::vector<char> hot(E, 0);
    double acc = 0.0;
    for (int e : order) {
        const double share = freq[e] / tot;
        if (acc + share > theta + 1e-9) break;
        acc += share;
        hot[e] = 1;
    }

    int S = 0;
    std::vector<int> seg_of_group(G, -1);
    for (int e = 0; e < E; ++e)
        if (hot[e]) {
            seg_kind[S] = 0;
            seg_id[S] = e;
            e2s[e] = S++;
        }
    for (int g = 0; g < G; ++g) {
        bool cold_member = false;
        for (int e = 0; e < E && !cold_member; ++e) cold_member = !hot[e] && e2g[e] == g;
        if (!cold_member) continue;
        seg_kind[S] = 1;
        seg_id[S] = g;
        seg_of_group[g] = S++;
    }
    for (int e = 0; e < E; ++e)
        if (!hot[e]) e2s[e] = seg_of_group[e2g[e]];
    *n_seg = S;
    return BMOE_OK;
}
