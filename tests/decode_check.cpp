// Host check of the work-item decode shared by the GEMM kernel and the host
// (kernel_params.h): over a grid of launch shapes and split settings chosen
// as the host chooses them, every work position maps to one (tile, K slice),
// every tile's slices cover its K exactly once with no empty slice, split
// counters and workspace tiles are distinct and within the launch's counts,
// and the tile-position walk visits every (row tile, column tile) once.
// Prints "ok <configurations>" or the first failure.
#include <cstdio>
#include <cstring>
#include <set>
#include <utility>
#include <vector>

#define __host__
#define __device__
#include "kernel_params.h"

using namespace compass;

static int round_slice(int K, int s) { return ((K + s - 1) / s + 63) / 64 * 64; }

static bool check(const GemmParams &p, char *why) {
    const int tiles = p.tiles_m * p.tiles_n;
    const int items = work_items(p);
    std::vector<std::vector<int>> cover(tiles);   // K coverage count per tile, in 64-deep steps
    std::vector<int> kseen(tiles, 0);
    std::set<int> counters, wstiles;
    std::set<std::pair<int, int>> seen;
    const int steps = (p.K + 63) / 64;
    for (int t = 0; t < tiles; ++t) cover[t].assign(steps, 0);
    int split_tiles = 0, ws_total = 0;
    for (int pos = 0; pos < items; ++pos) {
        const WorkItem w = decode_item(p, pos);
        if (w.tpos < 0 || w.tpos >= tiles) { std::sprintf(why, "pos %d: tile %d of %d", pos, w.tpos, tiles); return false; }
        if (w.slice < 0 || w.slice >= w.ns) { std::sprintf(why, "pos %d: slice %d of %d", pos, w.slice, w.ns); return false; }
        if (!seen.insert({w.tpos, w.slice}).second) { std::sprintf(why, "pos %d: (%d, %d) twice", pos, w.tpos, w.slice); return false; }
        const int kb = w.split ? w.slice * w.ksl : 0;
        const int ke = w.split ? (kb + w.ksl < p.K ? kb + w.ksl : p.K) : p.K;
        if (ke <= kb || kb % 64) { std::sprintf(why, "pos %d: K range [%d, %d)", pos, kb, ke); return false; }
        for (int k = kb / 64; k < (ke + 63) / 64; ++k) cover[w.tpos][k]++;
        kseen[w.tpos]++;
        if (w.split) {
            if (w.slice == 0) {
                if (!counters.insert(w.uc).second) { std::sprintf(why, "counter %d twice", w.uc); return false; }
                ++split_tiles;
                ws_total += w.ns;
            }
            if (!wstiles.insert(w.wsf + w.slice).second) { std::sprintf(why, "workspace tile %d twice", w.wsf + w.slice); return false; }
        }
    }
    for (int t = 0; t < tiles; ++t)
        for (int k = 0; k < steps; ++k)
            if (cover[t][k] != 1) { std::sprintf(why, "tile %d: K step %d covered %d times", t, k, cover[t][k]); return false; }
    for (int c : counters)
        if (c < 0 || c >= split_tiles) { std::sprintf(why, "counter %d outside [0, %d)", c, split_tiles); return false; }
    for (int x : wstiles)
        if (x < 0 || x >= ws_total) { std::sprintf(why, "workspace tile %d outside [0, %d)", x, ws_total); return false; }
    std::set<std::pair<int, int>> walk;
    for (int t = 0; t < tiles; ++t) {
        int ti, tn;
        tile_of(p, t, &ti, &tn);
        if (ti < 0 || ti >= p.tiles_m || tn < 0 || tn >= p.tiles_n || !walk.insert({ti, tn}).second) {
            std::sprintf(why, "tile position %d -> (%d, %d)", t, ti, tn);
            return false;
        }
    }
    return true;
}

int main() {
    int configs = 0;
    char why[256];
    const int tms[] = {1, 2, 3, 5, 8, 12, 32};
    const int tns[] = {1, 3, 24};
    const int gms[] = {1, 2, 4, 8};
    const int Ks[] = {64, 1000, 4096, 8192, 12288};
    for (int tm : tms)
        for (int tn : tns)
            for (int gm : gms)
                for (int K : Ks) {
                    const int groups = (tm + gm - 1) / gm;
                    const int gsz = gm * tn, tiles = tm * tn;
                    // head: whole leading groups, 2..4 slices of at least 2048 (as the host)
                    for (int hg = 0; hg <= groups; ++hg)
                        for (int hs = 2; hs <= 4; ++hs) {
                            const int head = hg < groups ? hg * gsz : tiles;
                            if (hg > 0 && K / hs < 2048) continue;
                            // tail: trailing groups from split_from, 2..4 slices (or none)
                            for (int tg = 0; tg <= groups - hg; ++tg)
                                for (int ts = 1; ts <= 4; ++ts) {
                                    if ((tg == 0) != (ts == 1)) continue;
                                    if (tg > 0 && K / ts < 2048) continue;
                                    GemmParams p;
                                    std::memset(&p, 0, sizeof p);
                                    p.tiles_m = tm;
                                    p.tiles_n = tn;
                                    p.group_m = gm;
                                    p.K = K;
                                    p.head_tiles = hg > 0 ? head : 0;
                                    p.head_split = hg > 0 ? hs : 0;
                                    p.head_kslice = hg > 0 ? round_slice(K, hs) : 0;
                                    p.ksplit = ts;
                                    p.kslice = ts > 1 ? round_slice(K, ts) : K;
                                    p.split_from = ts > 1 ? tiles - (tg * gsz < tiles ? tg * gsz : tiles) : p.head_tiles;
                                    if (p.split_from < p.head_tiles) continue;
                                    if (hg == 0 && hs > 2) continue;   // no head: one setting suffices
                                    ++configs;
                                    if (!check(p, why)) {
                                        std::printf("FAIL tm=%d tn=%d gm=%d K=%d head=%d/%d tail_from=%d/%d: %s\n", tm, tn,
                                                    gm, K, p.head_tiles, p.head_split, p.split_from, p.ksplit, why);
                                        return 1;
                                    }
                                }
                        }
                    // the general split (every tile, s slices of at least 512, s = ceil(K / slice))
                    for (int s = 2; s <= 16; ++s) {
                        if (K / s < 512) continue;
                        const int ks = round_slice(K, s);
                        const int sp = (K + ks - 1) / ks;
                        if (sp < 2) continue;
                        GemmParams p;
                        std::memset(&p, 0, sizeof p);
                        p.tiles_m = tm;
                        p.tiles_n = tn;
                        p.group_m = gm;
                        p.K = K;
                        p.ksplit = sp;
                        p.kslice = ks;
                        p.split_from = 0;
                        ++configs;
                        if (!check(p, why)) {
                            std::printf("FAIL general split tm=%d tn=%d K=%d s=%d: %s\n", tm, tn, K, sp, why);
                            return 1;
                        }
                    }
                }
    std::printf("ok %d\n", configs);
    return 0;
}
