/*
 * fp64 CPU oracle for the tiled Newton–Schulz map of Hierarchical Muon.
 *
 * TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py load this library. The HIP product path never
 * links, imports or calls it, and it shares no code, header, table or helper
 * with that path.
 *
 * Everything here is written straight from the paper's definitions, in
 * double precision, with plain loops and no blocking, fusion or reordering:
 *
 *   Sec. 2.2, eqs. (ns_iteration), (ns_quintic), (phi_k_def):
 *     for a nonzero H x W matrix A with H <= W,
 *       X_0     = A / ||A||_F
 *       X_{k+1} = (a I + b X_k X_k^T + c (X_k X_k^T)^2) X_k
 *       Phi_K(A) = X_K
 *     with I of size H x H. If H > W the recurrence runs on A^T and the
 *     result is transposed back. Phi_K(0) = 0.
 *
 *   Sec. 2.1 (Notation) and eq. (tiling_operator): the tiling operator B_T
 *     sets R = ceil(H/T), C = ceil(W/T), zero-pads A to (RT) x (CT) and cuts
 *     it into an R x C grid of T x T tiles; B_T^{-1} reassembles the tiles
 *     and drops the padding.
 *
 *   Sec. 4.1, eq. (tiled_ns):  Phi_{K,T}(A) = B_T^{-1}({Phi_K(A_rc)}).
 *
 * Every tile is therefore a full T x T (square) matrix, padding included,
 * exactly as the definition states; no orientation choice arises for tiles.
 * Tiles are numbered row-major over the grid: id = r*C + c.
 *
 * Status codes: 0 ok, -1 bad argument, -2 out of memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_BAD_ARG (-1)
#define ORACLE_NO_MEM (-2)

/* C (n x m) = P (n x q) * Q (q x m); all row-major and contiguous. */
static void matmul(const double* P, const double* Q, double* C, int64_t n, int64_t q, int64_t m)
{
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < m; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < q; ++k) s += P[i * q + k] * Q[k * m + j];
            C[i * m + j] = s;
        }
}

/* G (n x n) = X X^T for X (n x m). */
static void gram(const double* X, double* G, int64_t n, int64_t m)
{
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j) {
            double s = 0.0;
            for (int64_t k = 0; k < m; ++k) s += X[i * m + k] * X[j * m + k];
            G[i * n + j] = s;
        }
}

/* Row-oriented Phi_K for n <= m: X is n x m, overwritten with Phi_K(X). */
static int phi_k_rows(double* X, int64_t n, int64_t m, int K, double a, double b, double c)
{
    double nrm2 = 0.0;
    for (int64_t i = 0; i < n * m; ++i) nrm2 += X[i] * X[i];
    double nrm = sqrt(nrm2);
    if (nrm == 0.0) { /* Phi_K(0) = 0 */
        for (int64_t i = 0; i < n * m; ++i) X[i] = 0.0;
        return ORACLE_OK;
    }
    for (int64_t i = 0; i < n * m; ++i) X[i] = X[i] / nrm;

    double* A = (double*)malloc(sizeof(double) * n * n);  /* X X^T            */
    double* A2 = (double*)malloc(sizeof(double) * n * n); /* (X X^T)^2        */
    double* M = (double*)malloc(sizeof(double) * n * n);  /* aI + bA + cA^2   */
    double* Xn = (double*)malloc(sizeof(double) * n * m); /* M X              */
    if (!A || !A2 || !M || !Xn) {
        free(A); free(A2); free(M); free(Xn);
        return ORACLE_NO_MEM;
    }
    for (int k = 0; k < K; ++k) {
        gram(X, A, n, m);
        matmul(A, A, A2, n, n, n);
        for (int64_t i = 0; i < n; ++i)
            for (int64_t j = 0; j < n; ++j)
                M[i * n + j] = (i == j ? a : 0.0) + b * A[i * n + j] + c * A2[i * n + j];
        matmul(M, X, Xn, n, n, m);
        memcpy(X, Xn, sizeof(double) * n * m);
    }
    free(A); free(A2); free(M); free(Xn);
    return ORACLE_OK;
}

/*
 * Phi_K(A) for a dense H x W matrix (row-major, leading dimension ld_in),
 * written to Y (leading dimension ld_out). Applies the orientation rule of
 * Sec. 2.2: when H > W the recurrence runs on A^T and is transposed back.
 */
int oracle_phi_k(const double* A, int64_t H, int64_t W, int64_t ld_in, int K,
                 double a, double b, double c, double* Y, int64_t ld_out)
{
    if (!A || !Y || H < 1 || W < 1 || ld_in < W || ld_out < W || K < 0) return ORACLE_BAD_ARG;
    int transpose = H > W;
    int64_t n = transpose ? W : H, m = transpose ? H : W;
    double* X = (double*)malloc(sizeof(double) * n * m);
    if (!X) return ORACLE_NO_MEM;
    for (int64_t i = 0; i < H; ++i)
        for (int64_t j = 0; j < W; ++j) {
            if (transpose) X[j * m + i] = A[i * ld_in + j];
            else X[i * m + j] = A[i * ld_in + j];
        }
    int st = phi_k_rows(X, n, m, K, a, b, c);
    if (st == ORACLE_OK)
        for (int64_t i = 0; i < H; ++i)
            for (int64_t j = 0; j < W; ++j)
                Y[i * ld_out + j] = transpose ? X[j * m + i] : X[i * m + j];
    free(X);
    return st;
}

/* Number of tiles of B_T(A): R*C with R = ceil(H/T), C = ceil(W/T). */
int64_t oracle_tile_count(int64_t H, int64_t W, int64_t T)
{
    if (H < 1 || W < 1 || T < 1) return -1;
    int64_t R = (H + T - 1) / T, C = (W + T - 1) / T;
    return R * C;
}

/*
 * Rectangular tiles (T_h, T_w), used by the paper's tile-shape study (Sec.
 * 2.1 with T_h x T_w blocks in place of T x T): A is zero-padded to
 * (R T_h) x (C T_w), R = ceil(H/T_h), C = ceil(W/T_w), and cut into an R x C
 * grid of T_h x T_w tiles; square tiles are the case T_h = T_w = T.
 *
 * Phi_K of tile `tile_id` of that tiling, returned as the full T_h x T_w
 * tile Y (padding included, contiguous). Entry (i, j) of tile (r, c) is
 * A[r T_h + i][c T_w + j] when that lies inside A and 0 otherwise. A tile
 * with T_h > T_w goes through the orientation rule of oracle_phi_k.
 */
int oracle_ns_tile_hw(const double* A, int64_t H, int64_t W, int64_t ld_in, int64_t Th, int64_t Tw,
                      int64_t tile_id, int K, double a, double b, double c, double* Y)
{
    if (!A || !Y || H < 1 || W < 1 || ld_in < W || Th < 1 || Tw < 1 || K < 0) return ORACLE_BAD_ARG;
    int64_t R = (H + Th - 1) / Th, C = (W + Tw - 1) / Tw;
    if (tile_id < 0 || tile_id >= R * C) return ORACLE_BAD_ARG;
    int64_t r = tile_id / C, cc = tile_id % C;
    double* S = (double*)malloc(sizeof(double) * Th * Tw);
    if (!S) return ORACLE_NO_MEM;
    for (int64_t i = 0; i < Th; ++i)
        for (int64_t j = 0; j < Tw; ++j) {
            int64_t gi = r * Th + i, gj = cc * Tw + j;
            S[i * Tw + j] = (gi < H && gj < W) ? A[gi * ld_in + gj] : 0.0;
        }
    int st = oracle_phi_k(S, Th, Tw, Tw, K, a, b, c, Y, Tw);
    free(S);
    return st;
}

/* Phi_K of tile `tile_id` of B_T(A): the square case T_h = T_w = T. */
int oracle_ns_tile(const double* A, int64_t H, int64_t W, int64_t ld_in, int64_t T,
                   int64_t tile_id, int K, double a, double b, double c, double* Y)
{
    return oracle_ns_tile_hw(A, H, W, ld_in, T, T, tile_id, K, a, b, c, Y);
}

/*
 * The tiled map with T_h x T_w tiles: every tile through Phi_K, then the
 * tiles reassembled and the padding dropped, into Y (H x W, leading dim
 * ld_out). Tiles are independent; they are spread over OpenMP threads.
 */
int oracle_ns_tiled_hw(const double* A, int64_t H, int64_t W, int64_t ld_in, int64_t Th, int64_t Tw, int K,
                       double a, double b, double c, double* Y, int64_t ld_out)
{
    if (!A || !Y || H < 1 || W < 1 || ld_in < W || ld_out < W || Th < 1 || Tw < 1 || K < 0) return ORACLE_BAD_ARG;
    int64_t R = (H + Th - 1) / Th, C = (W + Tw - 1) / Tw;
    int status = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t t = 0; t < R * C; ++t) {
        double* Yt = (double*)malloc(sizeof(double) * Th * Tw);
        int st = Yt ? oracle_ns_tile_hw(A, H, W, ld_in, Th, Tw, t, K, a, b, c, Yt) : ORACLE_NO_MEM;
        if (st == ORACLE_OK) {
            int64_t r = t / C, cc = t % C;
            for (int64_t i = 0; i < Th; ++i)
                for (int64_t j = 0; j < Tw; ++j) {
                    int64_t gi = r * Th + i, gj = cc * Tw + j;
                    if (gi < H && gj < W) Y[gi * ld_out + gj] = Yt[i * Tw + j];
                }
        } else {
#pragma omp critical
            status = st;
        }
        free(Yt);
    }
    return status;
}

/*
 * Phi_{K,T}(A), eq. (tiled_ns): every tile of B_T(A) through Phi_K, then
 * B_T^{-1} (reassemble, drop the padding): the square case of the above.
 */
int oracle_ns_tiled(const double* A, int64_t H, int64_t W, int64_t ld_in, int64_t T, int K,
                    double a, double b, double c, double* Y, int64_t ld_out)
{
    return oracle_ns_tiled_hw(A, H, W, ld_in, T, T, K, a, b, c, Y, ld_out);
}

/*
 * A sample of tiles: Phi_K of tiles tile_ids[0..n_sel) of B_T(A), each
 * written as a full T x T tile at Y + s*T*T. Used where the whole matrix is
 * too large for the oracle to finish in seconds.
 */
int oracle_ns_tiles(const double* A, int64_t H, int64_t W, int64_t ld_in, int64_t T, int K,
                    double a, double b, double c, int64_t n_sel, const int64_t* tile_ids, double* Y)
{
    if (!tile_ids || n_sel < 0) return ORACLE_BAD_ARG;
    int status = ORACLE_OK;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t s = 0; s < n_sel; ++s) {
        int st = oracle_ns_tile(A, H, W, ld_in, T, tile_ids[s], K, a, b, c, Y + s * T * T);
        if (st != ORACLE_OK) {
#pragma omp critical
            status = st;
        }
    }
    return status;
}

/*
 * One HiMuon optimizer step of one matrix (Sec. 2.3's Muon update with the
 * tiled map substituted: Alg. 1 of Sec. 4.3, eq. (scaled_update) of Sec. 4.2), in place on
 * the H x W weights Wt and momentum Mt (both contiguous), given the gradient
 * G (contiguous):
 *   M   <- beta M + G                                   eq. (muon_momentum)
 *   Ghat = G + beta M  (Nesterov, eq. (muon_lookahead)), else Ghat = M
 *   if T == 0 (the branch T = infinity) or T >= max(H, W):
 *       U = Phi_K(Ghat),         tau = scale_c * sqrt(max(H, W))
 *   else
 *       U = Phi_{K,T}(Ghat),     tau = scale_c * sqrt(T)
 *   W   <- (1 - lr * lambda) W - lr * tau * U
 * The update direction U is also written to U_out when it is non-null.
 */
int oracle_himuon_step(double* Wt, double* Mt, const double* G, int64_t H, int64_t W, int64_t T, int K,
                       double a, double b, double c, double lr, double beta, double lambda, int nesterov,
                       double scale_c, double* U_out)
{
    if (!Wt || !Mt || !G || H < 1 || W < 1 || T < 0 || K < 0) return ORACLE_BAD_ARG;
    int64_t n = H * W;
    double* Ghat = (double*)malloc(sizeof(double) * n);
    double* U = (double*)malloc(sizeof(double) * n);
    if (!Ghat || !U) {
        free(Ghat);
        free(U);
        return ORACLE_NO_MEM;
    }
    for (int64_t i = 0; i < n; ++i) {
        Mt[i] = beta * Mt[i] + G[i];
        Ghat[i] = nesterov ? G[i] + beta * Mt[i] : Mt[i];
    }
    int64_t big = H > W ? H : W;
    int full = T == 0 || T >= big;
    int st = full ? oracle_phi_k(Ghat, H, W, W, K, a, b, c, U, W)
                  : oracle_ns_tiled(Ghat, H, W, W, T, K, a, b, c, U, W);
    if (st == ORACLE_OK) {
        double tau = scale_c * sqrt((double)(full ? big : T));
        for (int64_t i = 0; i < n; ++i) {
            Wt[i] = (1.0 - lr * lambda) * Wt[i] - lr * tau * U[i];
            if (U_out) U_out[i] = U[i];
        }
    }
    free(Ghat);
    free(U);
    return st;
}

/* Threads an OpenMP parallel region of this library uses (0 without OpenMP). */
int oracle_num_threads(void)
{
    int n = 0;
#pragma omp parallel
    {
#pragma omp atomic
        n += 1;
    }
    return n;
}
