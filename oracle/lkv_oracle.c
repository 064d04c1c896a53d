/*
 * CPU oracle for the linear-layer online prefill of LinearKV.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, fp64 statement of
 * what the GPU library computes.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no code, header or
 * constant with the GPU library, and the GPU library never calls it.
 *
 * Conventions (library form).  A recurrent layer's state for one value head is
 * S in R^{dv x dk}, row-major (dk contiguous).  The paper writes the state as
 * S_paper in R^{dk x dv} with S_i = T_i S_{i-1} + u_i (Eq. 1); the library
 * state is its transpose, S = S_paper^T, so the same recurrence reads
 *     S_t = S_{t-1} A_t + u_t^T,   A_t = T_t^T = T_t  (T_t is symmetric here).
 *
 *  - Gated DeltaNet (Eq. 3): A_t = alpha_t (I - beta_t k_t k_t^T),
 *    alpha_t = exp(g_t), u_t^T = beta_t v_t k_t^T (the delta-rule write of the
 *    cited GDN model), output o_t = scale * S_t q_t with the updated state.
 *  - Mamba-2 (Eq. 2): A_t = a_t I with the per-head scalar decay
 *    a_t = exp(dt_t A_h); u_t^T = dt_t x_t B_t^T; output y_t = S_t C_t.
 *  - Block summary (Eq. 5): a block maps an incoming state to
 *    S_out = S_in M + B, where B is the state the block reaches from zero and
 *    M = A_1 A_2 ... A_L (earliest token leftmost) is its transition.  Mamba-2
 *    keeps only the log-decay Lambda = A_h * sum_t dt_t (M = e^Lambda I).
 *  - Exact composition (Eq. 6): applying Eq. 5 block after block from an
 *    empty prefix, S <- S M_j + B_j for j = 1..K (M_1 is multiplied by zero and
 *    never read).
 *  - Single-block initialisation (Sec. 3.2): S_init = B_b for one block b.
 *
 * Arrays are packed "THD": [n_tok, heads, dim]; cu[s]..cu[s+1] are segment
 * s's tokens.  Value head h reads q/k head h / (h_v / h_qk).  All arithmetic
 * is fp64 on inputs widened exactly from their storage type.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

int lkvo_abi_version(void) { return 1; }

/* Gated DeltaNet, token by token (Eq. 1 and Eq. 3, library form).
 * S0 [n_seq,h_v,dv,dk] or NULL (zero start); o [n_tok,h_v,dv] or NULL;
 * S [n_seq,h_v,dv,dk] receives each segment's final state. */
void lkvo_gdn_scan(int64_t n_seq, const int32_t* cu, int h_qk, int h_v, int dk, int dv,
                   const double* q, const double* k, const double* v, const double* g,
                   const double* beta, double scale, const double* S0, double* o, double* S)
{
    const int group = h_v / h_qk;
    const int64_t n_pairs = n_seq * (int64_t)h_v;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pairs; ++p) {
        const int64_t s = p / h_v;
        const int h = (int)(p % h_v);
        const int hq = h / group;
        double* St = S + (size_t)p * dv * dk;
        if (S0) memcpy(St, S0 + (size_t)p * dv * dk, sizeof(double) * dv * dk);
        else memset(St, 0, sizeof(double) * dv * dk);
        for (int64_t t = cu[s]; t < cu[s + 1]; ++t) {
            const double* kt = k + ((size_t)t * h_qk + hq) * dk;
            const double* vt = v + ((size_t)t * h_v + h) * dv;
            const double alpha = exp(g[(size_t)t * h_v + h]);
            const double b = beta[(size_t)t * h_v + h];
            /* S <- S alpha (I - b k k^T) + b v k^T = alpha S + b (v - alpha S k) k^T */
            for (int i = 0; i < dv; ++i) {
                double* row = St + (size_t)i * dk;
                double sk = 0.0;
                for (int j = 0; j < dk; ++j) sk += row[j] * kt[j];
                const double d = b * (vt[i] - alpha * sk);
                for (int j = 0; j < dk; ++j) row[j] = alpha * row[j] + d * kt[j];
            }
            if (o) {
                const double* qt = q + ((size_t)t * h_qk + hq) * dk;
                double* ot = o + ((size_t)t * h_v + h) * dv;
                for (int i = 0; i < dv; ++i) {
                    const double* row = St + (size_t)i * dk;
                    double acc = 0.0;
                    for (int j = 0; j < dk; ++j) acc += row[j] * qt[j];
                    ot[i] = scale * acc;
                }
            }
        }
    }
}

/* Gated DeltaNet block transition M = A_1 ... A_L (Eq. 5, library form):
 * R <- I; for each token R <- R alpha (I - beta k k^T).  M [n_seq,h_v,dk,dk]. */
void lkvo_gdn_transition(int64_t n_seq, const int32_t* cu, int h_qk, int h_v, int dk,
                         const double* k, const double* g, const double* beta, double* M)
{
    const int group = h_v / h_qk;
    const int64_t n_pairs = n_seq * (int64_t)h_v;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pairs; ++p) {
        const int64_t s = p / h_v;
        const int h = (int)(p % h_v);
        const int hq = h / group;
        double* R = M + (size_t)p * dk * dk;
        memset(R, 0, sizeof(double) * dk * dk);
        for (int i = 0; i < dk; ++i) R[(size_t)i * dk + i] = 1.0;
        for (int64_t t = cu[s]; t < cu[s + 1]; ++t) {
            const double* kt = k + ((size_t)t * h_qk + hq) * dk;
            const double alpha = exp(g[(size_t)t * h_v + h]);
            const double b = beta[(size_t)t * h_v + h];
            for (int i = 0; i < dk; ++i) {
                double* row = R + (size_t)i * dk;
                double rk = 0.0;
                for (int j = 0; j < dk; ++j) rk += row[j] * kt[j];
                for (int j = 0; j < dk; ++j) row[j] = alpha * (row[j] - b * rk * kt[j]);
            }
        }
    }
}

/* Mamba-2 SSD, token by token (Eq. 1 and Eq. 2, library form), state S [P x N]:
 * a = exp(dt A_h); S <- a S + dt x B^T; y = S C.  C, B [n_tok,G,N]; x [n_tok,H,P];
 * dt [n_tok,H]; A [H]; S0/S [n_seq,H,P,N]; y [n_tok,H,P] or NULL. */
void lkvo_ssd_scan(int64_t n_seq, const int32_t* cu, int G, int H, int N, int P,
                   const double* C, const double* B, const double* x, const double* dt,
                   const double* A, const double* S0, double* y, double* S)
{
    const int group = H / G;
    const int64_t n_pairs = n_seq * (int64_t)H;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pairs; ++p) {
        const int64_t s = p / H;
        const int h = (int)(p % H);
        const int gi = h / group;
        double* St = S + (size_t)p * P * N;
        if (S0) memcpy(St, S0 + (size_t)p * P * N, sizeof(double) * P * N);
        else memset(St, 0, sizeof(double) * P * N);
        for (int64_t t = cu[s]; t < cu[s + 1]; ++t) {
            const double* Bt = B + ((size_t)t * G + gi) * N;
            const double* xt = x + ((size_t)t * H + h) * P;
            const double d = dt[(size_t)t * H + h];
            const double a = exp(d * A[h]);
            for (int i = 0; i < P; ++i) {
                double* row = St + (size_t)i * N;
                const double w = d * xt[i];
                for (int j = 0; j < N; ++j) row[j] = a * row[j] + w * Bt[j];
            }
            if (y) {
                const double* Ct = C + ((size_t)t * G + gi) * N;
                double* yt = y + ((size_t)t * H + h) * P;
                for (int i = 0; i < P; ++i) {
                    const double* row = St + (size_t)i * N;
                    double acc = 0.0;
                    for (int j = 0; j < N; ++j) acc += row[j] * Ct[j];
                    yt[i] = acc;
                }
            }
        }
    }
}

/* Mamba-2 block log-decay Lambda = A_h * sum_t dt_t (the scalar T_C of Eq. 5).
 * Lam [n_seq,H]. */
void lkvo_ssd_log_decay(int64_t n_seq, const int32_t* cu, int H, const double* dt,
                        const double* A, double* Lam)
{
    for (int64_t s = 0; s < n_seq; ++s)
        for (int h = 0; h < H; ++h) {
            double acc = 0.0;
            for (int64_t t = cu[s]; t < cu[s + 1]; ++t) acc += dt[(size_t)t * H + h];
            Lam[s * H + h] = A[h] * acc;
        }
}

/* Single-block initialisation (Sec. 3.2): S_init[r] = B_pool[src[r]], zeros for -1.
 * elems = per-request state size (heads * rows * cols). */
void lkvo_init_single(int32_t n_req, int64_t elems, const double* B_pool,
                      const int32_t* src, double* S_init)
{
    for (int32_t r = 0; r < n_req; ++r) {
        if (src[r] < 0) memset(S_init + (size_t)r * elems, 0, sizeof(double) * elems);
        else memcpy(S_init + (size_t)r * elems, B_pool + (size_t)src[r] * elems,
                    sizeof(double) * elems);
    }
}

/* Exact composition for Gated DeltaNet (Eq. 5 applied block after block, which
 * telescopes to Eq. 6): S <- 0; for each block j of the request in context
 * order, S <- S M_j + B_j.  The first block's M is multiplied by the zero state
 * and is not read.  B_pool [n_blk,h_v,dv,dk]; M_pool [n_blk,h_v,dk,dk];
 * S_init [n_req,h_v,dv,dk]. */
void lkvo_compose_gdn(int32_t n_req, const int32_t* blk_cu, const int32_t* blk_ids,
                      int h_v, int dv, int dk, const double* B_pool, const double* M_pool,
                      double* S_init)
{
    const int64_t n_pairs = (int64_t)n_req * h_v;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < n_pairs; ++p) {
        const int r = (int)(p / h_v);
        const int h = (int)(p % h_v);
        double* S = S_init + (size_t)p * dv * dk;
        double* tmp = (double*)malloc(sizeof(double) * dv * dk);
        memset(S, 0, sizeof(double) * dv * dk);
        for (int32_t e = blk_cu[r]; e < blk_cu[r + 1]; ++e) {
            const int32_t b = blk_ids[e];
            const double* Bj = B_pool + ((size_t)b * h_v + h) * dv * dk;
            if (e == blk_cu[r]) {
                memcpy(S, Bj, sizeof(double) * dv * dk);
                continue;
            }
            const double* Mj = M_pool + ((size_t)b * h_v + h) * dk * dk;
            for (int i = 0; i < dv; ++i)
                for (int j = 0; j < dk; ++j) {
                    double acc = 0.0;
                    for (int m = 0; m < dk; ++m) acc += S[(size_t)i * dk + m] * Mj[(size_t)m * dk + j];
                    tmp[(size_t)i * dk + j] = acc + Bj[(size_t)i * dk + j];
                }
            memcpy(S, tmp, sizeof(double) * dv * dk);
        }
        free(tmp);
    }
}

/* Exact composition for Mamba-2: S <- 0; S <- exp(Lambda_j) S + B_j per block.
 * B_pool [n_blk,H,P,N]; Lam_pool [n_blk,H]; S_init [n_req,H,P,N]. */
void lkvo_compose_ssd(int32_t n_req, const int32_t* blk_cu, const int32_t* blk_ids,
                      int H, int P, int N, const double* B_pool, const double* Lam_pool,
                      double* S_init)
{
    const size_t st = (size_t)P * N;
    for (int32_t r = 0; r < n_req; ++r)
        for (int h = 0; h < H; ++h) {
            double* S = S_init + ((size_t)r * H + h) * st;
            memset(S, 0, sizeof(double) * st);
            for (int32_t e = blk_cu[r]; e < blk_cu[r + 1]; ++e) {
                const int32_t b = blk_ids[e];
                const double* Bj = B_pool + ((size_t)b * H + h) * st;
                const double a = (e == blk_cu[r]) ? 0.0 : exp(Lam_pool[(size_t)b * H + h]);
                for (size_t i = 0; i < st; ++i) S[i] = (e == blk_cu[r]) ? Bj[i] : a * S[i] + Bj[i];
            }
        }
}
