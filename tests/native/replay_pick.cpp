// Host check of the row-selection rule that ends a stage-1 group replay (replay_pick_* in verify.hpp): the
// lowest row whose replayed score equals the stage-1 score; failing that, the lowest row at the replay's own
// maximum, reported as a fallback; -1 when no row was offered.  The rows of a 16-row group are offered in
// four lane-sized pieces merged in every order, as the wave merges them.  Exits non-zero on the first failure.
#include <algorithm>
#include <cstdio>
#include <random>
#include <vector>

#include "verify.hpp"

using namespace lacache;

// the rule written out directly
static int want_row(const std::vector<float>& v, const std::vector<int>& rows, float s, bool* fb) {
    int exact = -1, top = -1;
    for (size_t i = 0; i < v.size(); ++i) {
        if (v[i] == s && (exact < 0 || rows[i] < exact)) exact = rows[i];
        if (top < 0 || v[i] > v[std::find(rows.begin(), rows.end(), top) - rows.begin()] ||
            (v[i] == v[std::find(rows.begin(), rows.end(), top) - rows.begin()] && rows[i] < top))
            top = rows[i];
    }
    *fb = exact < 0;
    return exact >= 0 ? exact : top;
}

static int got_row(const std::vector<float>& v, const std::vector<int>& rows, float s, bool* fb, int order) {
    // four lanes of four rows each, merged in the order given by `order` (a permutation index)
    ReplayPick part[4];
    for (int l = 0; l < 4; ++l) part[l] = replay_pick_none();
    for (size_t i = 0; i < v.size(); ++i) part[i % 4] = replay_pick_add(part[i % 4], rows[i], v[i], s);
    int perm[4] = {0, 1, 2, 3};
    for (int k = 0; k < order; ++k) std::next_permutation(perm, perm + 4);
    ReplayPick p = part[perm[0]];
    for (int l = 1; l < 4; ++l) p = replay_pick_merge(p, part[perm[l]]);
    return replay_pick_row(p, fb);
}

int main() {
    std::mt19937 rng(7);
    long cases = 0;
    for (int t = 0; t < 200000; ++t) {
        const int n = 1 + (int)(rng() % 16);                   // valid rows of the group
        std::vector<int> rows(n);
        const int g0 = (int)(rng() % 1000) * 16;
        for (int i = 0; i < n; ++i) rows[i] = g0 + i;
        std::shuffle(rows.begin(), rows.end(), rng);          // lanes see rows in any order
        std::vector<float> v(n);
        const int levels = 1 + (int)(rng() % 4);               // few distinct values: many exact ties
        for (int i = 0; i < n; ++i) v[i] = (float)(rng() % levels) * 0.25f - 0.5f;
        float s;
        switch (rng() % 3) {
            case 0: s = *std::max_element(v.begin(), v.end()); break;   // the usual case: the maximum
            case 1: s = v[rng() % n]; break;                            // any present value
            default: s = 7.0f; break;                                   // absent: the fallback
        }
        bool fw, fg;
        const int w = want_row(v, rows, s, &fw);
        const int g = got_row(v, rows, s, &fg, (int)(rng() % 24));
        ++cases;
        if (w != g || fw != fg) {
            std::printf("MISMATCH case %d: want row %d (fallback %d), got %d (fallback %d)\n", t, w, (int)fw, g,
                        (int)fg);
            return 1;
        }
    }
    // no row offered: -1, flagged
    bool fb = false;
    if (replay_pick_row(replay_pick_none(), &fb) != -1 || !fb) {
        std::printf("MISMATCH: an empty pick must name no row\n");
        return 1;
    }
    std::printf("ok %ld cases\n", cases);
    return 0;
}
