/*
 * Oracle neighbour list -- TEST INFRASTRUCTURE ONLY.
 *
 * Brute-force definition of the neighbour set of Methods, "The neighbor
 * graph", Eq. (neighbor-set):  N_i = { (j, n) : |r_j + n.h - r_i| < r,
 * (j, n) != (i, 0) }, with every periodic image n a distinct instance and
 * both orientations of a pair stored.
 *
 * Exact predicate.  Positions and lattice vectors are mapped to 64-bit fixed
 * point, Q(x) = nearest integer of x * 2^20 (ties to even), and the test
 * |Q(r_j) + sum_a n_a Q(h_a) - Q(r_i)|^2 < Q(r)^2 is evaluated in integer
 * arithmetic, so the list is a deterministic function of the float64 input.
 * The fixed-point boundary differs from the real one only within ~1e-6 A of
 * r, where the smooth envelope of Eq. (envelope) is ~1e-27.
 *
 * Output order is canonical: ascending (i, j, n_x, n_y, n_z).  The loops
 * below run in exactly that order, so no sort is needed.
 *
 * Every centre i in ``centres`` (or all centres when centres == NULL) is
 * compared with every atom j and every image n in a range that is proven
 * wide enough from the fractional displacement (see image_range); nothing
 * else is pruned.  O(N_centres * N * images): meant for small systems and for
 * sampled centres of large ones.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define QSCALE 1048576.0 /* 2^20 */

static int64_t q_of(double x) { return (int64_t)llrint(x * QSCALE); }

/* Inverse of a 3x3 matrix with rows h_a (returns 0 if singular). */
static int inv3(const double h[9], double out[9]) {
    double a = h[0], b = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], k = h[7], l = h[8];
    double det = a * (e * l - f * k) - b * (d * l - f * g) + c * (d * k - e * g);
    if (det == 0.0) return 0;
    out[0] = (e * l - f * k) / det; out[1] = (c * k - b * l) / det; out[2] = (b * f - c * e) / det;
    out[3] = (f * g - d * l) / det; out[4] = (a * l - c * g) / det; out[5] = (c * d - a * f) / det;
    out[6] = (d * k - e * g) / det; out[7] = (b * g - a * k) / det; out[8] = (a * e - b * d) / det;
    return 1;
}

/*
 * Image range along axis a.  Write r_j - r_i = f.h (f fractional).  Any image
 * with |(f + n).h| < r' has |f_a + n_a| < r' |b_a|, where b_a is the a-th
 * reciprocal vector (column a of h^-1), because (f+n)_a = ((f+n).h) . b_a.
 * r' = r + 1e-3 A covers the fixed-point rounding of positions and lattice
 * vectors (<= (2 + 3|n|) sqrt(3) 2^-21 A, i.e. < 1e-3 A for |n| < 1000) and
 * float rounding in f; the integer predicate then decides membership exactly.
 */
static void image_range(double fa, double reach, int periodic, int64_t* lo, int64_t* hi) {
    if (!periodic) { *lo = 0; *hi = 0; return; }
    *lo = (int64_t)ceil(-fa - reach);
    *hi = (int64_t)floor(-fa + reach);
}

/*
 * pos     [n][3] float64        cell [3][3] rows = lattice vectors
 * pbc     [3] int               r    cutoff (Angstrom)
 * centres [n_centres] int64 or NULL (all atoms, in order)
 * Output arrays have capacity ``cap``; *n_out receives the number of edges
 * even when it exceeds cap (then nothing beyond cap is written, return 1).
 * Returns 0 on success, 1 on capacity overflow, 2 on bad input.
 */
int oracle_neighbors_brute(const double* pos, int64_t n, const double* cell, const int* pbc,
                           double r, const int64_t* centres, int64_t n_centres, int64_t cap,
                           int64_t* out_i, int32_t* out_j, int32_t* out_n, int64_t* n_out) {
    double hinv[9];
    if (!inv3(cell, hinv)) return 2;
    int64_t qh[9];
    for (int k = 0; k < 9; ++k) qh[k] = q_of(cell[k]);
    int64_t qr = q_of(r);
    /* |b_a| = norm of column a of h^-1 */
    double reach[3];
    for (int a = 0; a < 3; ++a) {
        double s = hinv[0 * 3 + a] * hinv[0 * 3 + a] + hinv[1 * 3 + a] * hinv[1 * 3 + a] +
                   hinv[2 * 3 + a] * hinv[2 * 3 + a];
        reach[a] = (r + 1.0e-3) * sqrt(s);
    }
    int64_t count = 0;
    int64_t nc = centres ? n_centres : n;
    for (int64_t ci = 0; ci < nc; ++ci) {
        int64_t i = centres ? centres[ci] : ci;
        if (i < 0 || i >= n) return 2;
        int64_t qi[3] = {q_of(pos[3 * i]), q_of(pos[3 * i + 1]), q_of(pos[3 * i + 2])};
        for (int64_t j = 0; j < n; ++j) {
            int64_t qj[3] = {q_of(pos[3 * j]), q_of(pos[3 * j + 1]), q_of(pos[3 * j + 2])};
            double d[3] = {pos[3 * j] - pos[3 * i], pos[3 * j + 1] - pos[3 * i + 1],
                           pos[3 * j + 2] - pos[3 * i + 2]};
            double f[3];
            for (int a = 0; a < 3; ++a)
                f[a] = d[0] * hinv[0 * 3 + a] + d[1] * hinv[1 * 3 + a] + d[2] * hinv[2 * 3 + a];
            int64_t lo[3], hi[3];
            for (int a = 0; a < 3; ++a) image_range(f[a], reach[a], pbc[a], &lo[a], &hi[a]);
            for (int64_t nx = lo[0]; nx <= hi[0]; ++nx)
                for (int64_t ny = lo[1]; ny <= hi[1]; ++ny)
                    for (int64_t nz = lo[2]; nz <= hi[2]; ++nz) {
                        if (j == i && nx == 0 && ny == 0 && nz == 0) continue;
                        int64_t dq[3];
                        int far = 0;
                        for (int a = 0; a < 3; ++a) {
                            dq[a] = qj[a] + nx * qh[0 * 3 + a] + ny * qh[1 * 3 + a] +
                                    nz * qh[2 * 3 + a] - qi[a];
                            if (dq[a] >= qr || dq[a] <= -qr) far = 1; /* avoids overflow */
                        }
                        if (far) continue;
                        __int128 d2 = (__int128)dq[0] * dq[0] + (__int128)dq[1] * dq[1] +
                                      (__int128)dq[2] * dq[2];
                        if (d2 >= (__int128)qr * qr) continue;
                        if (count < cap) {
                            out_i[count] = i;
                            out_j[count] = (int32_t)j;
                            out_n[3 * count + 0] = (int32_t)nx;
                            out_n[3 * count + 1] = (int32_t)ny;
                            out_n[3 * count + 2] = (int32_t)nz;
                        }
                        ++count;
                    }
        }
    }
    *n_out = count;
    return count > cap ? 1 : 0;
}
