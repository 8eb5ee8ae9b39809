// Workgroup -> output tile order of the bf16 GEMM (shared by the kernel and its host-side
// dispatcher; plain C++ so that a host compiler can check the mapping as well).
//
// The GPU hands workgroup b to XCD b % 8 as that XCD's (b / 8)-th workgroup, and each XCD
// has an L2 of its own.  The tiles are put in one global order and XCD x takes the x-th
// eighth of it, so the workgroups that run together on one XCD are neighbours in that order
// and share operand rows in its L2.  The global order walks the tile grid (nt_m row tiles by
// nt_n column tiles) in bands of `band` row tiles: band after band, within a band column after
// column, rows fastest within a column.  A last, shorter band takes the remaining rows.
// band = nt_m is one whole column after another (every row tile of a weight tile on one XCD,
// right for few row tiles); a short band keeps a few activation row tiles and a few weight
// tiles in each XCD's working set when there are many row tiles.
#ifndef SGD_TILE_ORDER_H
#define SGD_TILE_ORDER_H

#ifdef __HIPCC__
#define SGD_HD __host__ __device__
#else
#define SGD_HD
#endif

namespace sgd {

constexpr int kXcds = 8;         // XCDs of the GPU, dispatched round-robin
constexpr int kCusPerXcd = 32;   // one workgroup per CU: the workgroups running at once on an XCD

// position of workgroup bid in the global order
SGD_HD inline int tile_position(int bid, int total) {
    if (total % kXcds) return bid;
    return (bid % kXcds) * (total / kXcds) + bid / kXcds;
}

// tile (row tile tm, column tile tn) at position pos of the banded order
SGD_HD inline void tile_at(int pos, int nt_m, int nt_n, int band, int& tm, int& tn) {
    if (band <= 0 || band > nt_m) band = nt_m;
    const int b = pos / (band * nt_n);
    const int rows = nt_m - b * band < band ? nt_m - b * band : band;  // rows of this band
    const int r = pos - b * band * nt_n;
    tm = b * band + r % rows;
    tn = r / rows;
}

// Band for a launch: the smallest operand footprint (activation rows x BM + weight rows x BN)
// of the kCusPerXcd workgroups that run together on one XCD; ties keep the larger band.  Grids
// that do not split evenly over the XCDs keep whole columns.
inline int tile_band(int nt_m, int nt_n, int bm, int bn) {
    if ((nt_m * nt_n) % kXcds) return nt_m;
    int best = nt_m;
    long best_fp = -1;
    for (int band = nt_m; band >= 1; band = band > 1 ? (band + 1) / 2 : 0) {
        const int rows = band < kCusPerXcd ? band : kCusPerXcd;
        int cols = (kCusPerXcd + rows - 1) / rows;
        if (cols > nt_n) cols = nt_n;
        const long fp = (long)rows * bm + (long)cols * bn;
        if (best_fp < 0 || fp < best_fp) { best_fp = fp; best = band; }
        if (band == 1) break;
    }
    return best;
}

}  // namespace sgd

#endif  // SGD_TILE_ORDER_H
