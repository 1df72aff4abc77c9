/*
 * YOSO attention: plain, slow CPU oracle in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link or
 * call this file; only the tests, the smoke check and the CPU baseline of the
 * bench use it.  It shares no code with the HIP path.
 *
 * Every routine follows the paper's text (You Only Sample (Almost) Once,
 * arXiv 2111.09714) step by step, with the obvious loops and no blocking:
 *
 *   hash        Sec. 3.2 overview + Fig. 2 caption: a code is tau concatenated
 *               random-hyperplane (sign) hashes; m independent hashes.
 *   forward     Sec. 3.2 overview: per hash, a table of 2^tau d-vectors holds the
 *               sum of the values whose key falls in each bucket; a query reads
 *               the bucket of its own code.  Sec. 3.1: the output is the average
 *               over the m hashes.
 *   backward    Sec. 3.3: eq. (gradient-v) for dV (the table machinery with the
 *               roles of queries and keys swapped); eq. (pseudo-gradient-q) for the
 *               lower-bound surrogate dQ evaluated on the sampled B, and the
 *               symmetric expression for dK; all averaged over the m hashes.
 *   backward_d2 the same surrogate written as eq. (backward-d2): d runs of the
 *               bucket-table subroutine, used to cross-check the pairwise form.
 *   backward_star  *YOSO (Sec. 3.3 eq. (gradient-q); Sec. 4): an unbiased
 *               sampled estimate of the true gradient on the same hashes, from
 *               the pairs whose codes agree on all bits but at most one.
 *   expectation eq. (yoso-expectation): E[B_ij] = (1 - arccos(q_i.k_j)/pi)^tau,
 *               giving E[Y], E[dV], E[dQ], E[dK], and the true dQ of
 *               eq. (gradient-q) for reference.
 *   l2_normalize          Sec. 3.1 "Normalizing Attention" (eq. normalized-yoso:
 *               N-YOSO = l2(B V)) and Sec. 4 (Q, K l2-normalised before hashing):
 *               each row divided by its Euclidean norm.
 *   l2_normalize_backward the Jacobian of that map, built entry by entry and
 *               applied to the incoming gradient (no simplification).
 *   fast_hyperplanes  Sec. 3.2 "Speed-up": the approximate random projection of
 *               Andoni et al. (2015), a pseudo-random rotation H D3 H D2 H D1 (H the
 *               Walsh-Hadamard matrix, D_i random +-1 diagonals).  Its rows are the
 *               hyperplanes of the fast hash; the routine writes them out as an
 *               ordinary R for the hash routine above, by dense matrix products.
 *
 * Conventions (readings of points the paper leaves open):
 *   - bit b of hash h is [ sum_l x_l R[l][h*tau+b] > 0 ] (strict), code = sum_b bit_b 2^b;
 *   - the same hyperplanes hash queries and keys; the backward reuses the
 *     forward's codes;
 *   - m-hash averaging is the arithmetic mean, applied to Y, dV, dQ, dK;
 *   - empty buckets contribute 0 (no renormalisation);
 *   - l2 normalisation maps the zero row to the zero row, with zero gradient;
 *   - tensors are row-major: x[bh][i][l], codes[bh][h][i];
 *   - fast hash: rotation r supplies the hyperplanes of columns r*d .. r*d+d-1 of
 *     R in order (column c = h*tau + b is row c mod d of rotation c / d), and
 *     bit l of signs[3r + i] set means D_{i+1} of rotation r negates coordinate l;
 *     the rotation is scaled by 1/d so that each row has length sqrt(d), as a
 *     column of a standard Gaussian R has on average (signs do not depend on it).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define CODE(codes, b, h, i, m, n) ((codes)[(((int64_t)(b) * (m) + (h)) * (n)) + (i)])

/* Sign-random-projection hash.  x: [bh][n][d], R: [d][m*tau].
 * codes: [bh][m][n]; minabs (optional): [bh][m][n], the smallest |projection|
 * over the tau hyperplanes of each (row, hash), used to tell which bits sit so
 * close to a hyperplane that rounding may flip them. */
void oracle_hash(const double *x, int64_t bh, int64_t n, int d,
                 const double *R, int m, int tau,
                 uint16_t *codes, double *minabs)
{
    const int ncol = m * tau;
    for (int64_t b = 0; b < bh; b++) {
        for (int64_t i = 0; i < n; i++) {
            const double *row = x + (b * n + i) * d;
            for (int h = 0; h < m; h++) {
                unsigned code = 0;
                double closest = INFINITY;
                for (int bit = 0; bit < tau; bit++) {
                    const int col = h * tau + bit;
                    double s = 0.0;
                    for (int l = 0; l < d; l++)
                        s += row[l] * R[(int64_t)l * ncol + col];
                    if (s > 0.0)
                        code |= 1u << bit;
                    if (fabs(s) < closest)
                        closest = fabs(s);
                }
                CODE(codes, b, h, i, m, n) = (uint16_t)code;
                if (minabs)
                    CODE(minabs, b, h, i, m, n) = closest;
            }
        }
    }
}

/* One run of the bucket-table subroutine for a single (head, hash):
 * table[c] = sum over sources s with src_code[s] == c of val[s]   (width w)
 * out[t]  += weight * table[dst_code[t]]                          for every target t
 * This is the scatter/gather of the Sec. 3.2 overview. */
static void table_pass(const uint16_t *src_code, const double *val, int64_t n_src,
                       const uint16_t *dst_code, int64_t n_dst, int w, int tau,
                       double weight, double *out, double *table)
{
    const int64_t buckets = (int64_t)1 << tau;
    memset(table, 0, sizeof(double) * buckets * w);
    for (int64_t s = 0; s < n_src; s++)
        for (int l = 0; l < w; l++)
            table[(int64_t)src_code[s] * w + l] += val[s * w + l];
    for (int64_t t = 0; t < n_dst; t++)
        for (int l = 0; l < w; l++)
            out[t * w + l] += weight * table[(int64_t)dst_code[t] * w + l];
}

/* Forward: y[bh][i] = (1/m) sum_h sum_{j : kc_h(j) == qc_h(i)} v[bh][j]. */
void oracle_forward(const uint16_t *qc, const uint16_t *kc, const double *v,
                    int64_t bh, int64_t nq, int64_t nk, int d, int m, int tau,
                    double *y)
{
    double *table = malloc(sizeof(double) * ((size_t)1 << tau) * d);
    memset(y, 0, sizeof(double) * bh * nq * d);
    for (int64_t b = 0; b < bh; b++)
        for (int h = 0; h < m; h++)
            table_pass(&CODE(kc, b, h, 0, m, nk), v + b * nk * d, nk,
                       &CODE(qc, b, h, 0, m, nq), nq, d, tau, 1.0 / m,
                       y + b * nq * d, table);
    free(table);
}

/* Backward.
 * dv = (1/m) sum_h B_h^T dy                        (eq. gradient-v, sampled form)
 * dq = tau/(2m) sum_h [(dy v^T) .* B_h] k          (eq. pseudo-gradient-q, sampled)
 * dk = tau/(2m) sum_h [(dy v^T) .* B_h]^T q        (the symmetric expression)
 * dQ/dK are evaluated bucket by bucket over colliding pairs. */
void oracle_backward(const uint16_t *qc, const uint16_t *kc,
                     const double *q, const double *k, const double *v, const double *dy,
                     int64_t bh, int64_t nq, int64_t nk, int d, int m, int tau,
                     double *dq, double *dk, double *dv)
{
    const int64_t buckets = (int64_t)1 << tau;
    double *table = malloc(sizeof(double) * buckets * d);
    /* bucket membership lists: start[c] .. start[c+1] index into members */
    int64_t *qstart = malloc(sizeof(int64_t) * (buckets + 1));
    int64_t *kstart = malloc(sizeof(int64_t) * (buckets + 1));
    int64_t *qmem = malloc(sizeof(int64_t) * (nq > 0 ? nq : 1));
    int64_t *kmem = malloc(sizeof(int64_t) * (nk > 0 ? nk : 1));
    int64_t *fill = malloc(sizeof(int64_t) * buckets);
    const double scale = (double)tau / (2.0 * m);

    memset(dq, 0, sizeof(double) * bh * nq * d);
    memset(dk, 0, sizeof(double) * bh * nk * d);
    memset(dv, 0, sizeof(double) * bh * nk * d);

    for (int64_t b = 0; b < bh; b++) {
        const double *qb = q + b * nq * d, *kb = k + b * nk * d;
        const double *vb = v + b * nk * d, *dyb = dy + b * nq * d;
        double *dqb = dq + b * nq * d, *dkb = dk + b * nk * d;
        for (int h = 0; h < m; h++) {
            const uint16_t *qch = &CODE(qc, b, h, 0, m, nq);
            const uint16_t *kch = &CODE(kc, b, h, 0, m, nk);

            /* dV: table of dy keyed by query codes, read at key codes. */
            table_pass(qch, dyb, nq, kch, nk, d, tau, 1.0 / m, dv + b * nk * d, table);

            /* Group rows by bucket (a plain counting sort). */
            for (int64_t c = 0; c <= buckets; c++) qstart[c] = kstart[c] = 0;
            for (int64_t i = 0; i < nq; i++) qstart[qch[i] + 1]++;
            for (int64_t j = 0; j < nk; j++) kstart[kch[j] + 1]++;
            for (int64_t c = 0; c < buckets; c++) {
                qstart[c + 1] += qstart[c];
                kstart[c + 1] += kstart[c];
            }
            for (int64_t c = 0; c < buckets; c++) fill[c] = qstart[c];
            for (int64_t i = 0; i < nq; i++) qmem[fill[qch[i]]++] = i;
            for (int64_t c = 0; c < buckets; c++) fill[c] = kstart[c];
            for (int64_t j = 0; j < nk; j++) kmem[fill[kch[j]]++] = j;

            /* Every colliding pair (i, j): s = dy_i . v_j,
             * dq_i += scale * s * k_j,  dk_j += scale * s * q_i. */
            for (int64_t c = 0; c < buckets; c++) {
                for (int64_t a = qstart[c]; a < qstart[c + 1]; a++) {
                    const int64_t i = qmem[a];
                    for (int64_t e = kstart[c]; e < kstart[c + 1]; e++) {
                        const int64_t j = kmem[e];
                        double s = 0.0;
                        for (int l = 0; l < d; l++)
                            s += dyb[i * d + l] * vb[j * d + l];
                        for (int l = 0; l < d; l++) {
                            dqb[i * d + l] += scale * s * kb[j * d + l];
                            dkb[j * d + l] += scale * s * qb[i * d + l];
                        }
                    }
                }
            }
        }
    }
    free(table); free(qstart); free(kstart); free(qmem); free(kmem); free(fill);
}

/* *YOSO: a sampled estimate of the TRUE gradient of eq. (gradient-q) and of its
 * symmetric counterpart for K, on the same m hashes (Sec. 3.3; the variant the
 * experiments call *YOSO, Sec. 4).
 *
 * eq. (gradient-q) weighs the pair (i, j) by tau (1 - theta_ij/pi)^(tau-1) /
 * (pi sqrt(1 - x_ij^2)), x_ij = q_i . k_j, theta_ij = arccos x_ij.  The factor
 * (1 - theta/pi)^(tau-1) is the probability that tau-1 independent hyperplane
 * bits agree (the collision law of the Fig. 2 caption with one bit fewer).  A
 * tau-bit code minus its bit t is such a (tau-1)-bit hash, so for every hash h
 *
 *   C_h(i, j) = sum_{t < tau} [ codes of q_i and k_j agree on every bit except t ]
 *
 * has expectation tau (1 - theta_ij/pi)^(tau-1), and
 *
 *   dq_i = (1/m) sum_h sum_j C_h(i, j) (dy_i . v_j) / (pi sqrt(max(1 - x_ij^2, eps))) k_j
 *   dk_j = (1/m) sum_h sum_i C_h(i, j) (dy_i . v_j) / (pi sqrt(max(1 - x_ij^2, eps))) q_i
 *
 * is unbiased for eq. (gradient-q) wherever 1 - x^2 >= eps.  The paper notes
 * that the true gradient diverges as the alignment x approaches 1; eps = `floor`
 * bounds the weight (floor = 0: no bound).  x is the dot product of the rows as
 * given, clamped to [-1, 1] (the method takes unit rows).  dv is eq. (gradient-v)
 * exactly as in oracle_backward. */
void oracle_backward_star(const uint16_t *qc, const uint16_t *kc,
                          const double *q, const double *k, const double *v, const double *dy,
                          int64_t bh, int64_t nq, int64_t nk, int d, int m, int tau, double floor_,
                          double *dq, double *dk, double *dv)
{
    const int64_t buckets = (int64_t)1 << tau;
    const unsigned full = (unsigned)buckets - 1u;
    double *table = malloc(sizeof(double) * buckets * d);

    memset(dq, 0, sizeof(double) * bh * nq * d);
    memset(dk, 0, sizeof(double) * bh * nk * d);
    memset(dv, 0, sizeof(double) * bh * nk * d);

    for (int64_t b = 0; b < bh; b++) {
        const double *qb = q + b * nq * d, *kb = k + b * nk * d;
        const double *vb = v + b * nk * d, *dyb = dy + b * nq * d;
        double *dqb = dq + b * nq * d, *dkb = dk + b * nk * d;
        for (int h = 0; h < m; h++) {
            const uint16_t *qch = &CODE(qc, b, h, 0, m, nq);
            const uint16_t *kch = &CODE(kc, b, h, 0, m, nk);
            table_pass(qch, dyb, nq, kch, nk, d, tau, 1.0 / m, dv + b * nk * d, table);
            for (int64_t i = 0; i < nq; i++) {
                for (int64_t j = 0; j < nk; j++) {
                    /* the dropped-bit hashes under which i and j collide */
                    int count = 0;
                    for (int t = 0; t < tau; t++) {
                        const unsigned keep = full & ~(1u << t);
                        if (((qch[i] ^ kch[j]) & keep) == 0) count++;
                    }
                    if (count == 0) continue;
                    double s = 0.0, x = 0.0;
                    for (int l = 0; l < d; l++) {
                        s += dyb[i * d + l] * vb[j * d + l];
                        x += qb[i * d + l] * kb[j * d + l];
                    }
                    if (x > 1.0) x = 1.0;
                    if (x < -1.0) x = -1.0;
                    double r = 1.0 - x * x;
                    if (r < floor_) r = floor_;
                    const double w = count / (M_PI * sqrt(r)) / m;
                    for (int l = 0; l < d; l++) {
                        dqb[i * d + l] += w * s * kb[j * d + l];
                        dkb[j * d + l] += w * s * qb[i * d + l];
                    }
                }
            }
        }
    }
    free(table);
}

/* The same dQ, dK surrogate in the form of eq. (backward-d2):
 *   dq_i = (1/m) sum_h sum_l dy_{i,l} sum_j B_h(i,j) (v_{j,l} (tau/2) k_j)
 * i.e. for every value dimension l one bucket-table run whose table rows are
 * the d-vectors v_{j,l} (tau/2) k_j, read at the query codes and weighted by
 * dy_{i,l}.  dk is the mirror image: tables of dy_{i,l} (tau/2) q_i keyed by the
 * query codes, read at the key codes and weighted by v_{j,l}. */
void oracle_backward_d2(const uint16_t *qc, const uint16_t *kc,
                        const double *q, const double *k, const double *v, const double *dy,
                        int64_t bh, int64_t nq, int64_t nk, int d, int m, int tau,
                        double *dq, double *dk)
{
    const int64_t buckets = (int64_t)1 << tau;
    double *table = malloc(sizeof(double) * buckets * d);
    double *rows = malloc(sizeof(double) * (nq > nk ? nq : nk) * d + 1);
    double *part = malloc(sizeof(double) * (nq > nk ? nq : nk) * d + 1);
    memset(dq, 0, sizeof(double) * bh * nq * d);
    memset(dk, 0, sizeof(double) * bh * nk * d);
    for (int64_t b = 0; b < bh; b++) {
        const double *qb = q + b * nq * d, *kb = k + b * nk * d;
        const double *vb = v + b * nk * d, *dyb = dy + b * nq * d;
        for (int h = 0; h < m; h++) {
            const uint16_t *qch = &CODE(qc, b, h, 0, m, nq);
            const uint16_t *kch = &CODE(kc, b, h, 0, m, nk);
            for (int l = 0; l < d; l++) {
                /* dQ: table rows v_{j,l} (tau/2) k_j keyed by key codes. */
                for (int64_t j = 0; j < nk; j++)
                    for (int e = 0; e < d; e++)
                        rows[j * d + e] = vb[j * d + l] * (tau / 2.0) * kb[j * d + e];
                memset(part, 0, sizeof(double) * nq * d);
                table_pass(kch, rows, nk, qch, nq, d, tau, 1.0, part, table);
                for (int64_t i = 0; i < nq; i++)
                    for (int e = 0; e < d; e++)
                        dq[(b * nq + i) * d + e] += dyb[i * d + l] * part[i * d + e] / m;
                /* dK: table rows dy_{i,l} (tau/2) q_i keyed by query codes. */
                for (int64_t i = 0; i < nq; i++)
                    for (int e = 0; e < d; e++)
                        rows[i * d + e] = dyb[i * d + l] * (tau / 2.0) * qb[i * d + e];
                memset(part, 0, sizeof(double) * nk * d);
                table_pass(qch, rows, nq, kch, nk, d, tau, 1.0, part, table);
                for (int64_t j = 0; j < nk; j++)
                    for (int e = 0; e < d; e++)
                        dk[(b * nk + j) * d + e] += vb[j * d + l] * part[j * d + e] / m;
            }
        }
    }
    free(table); free(rows); free(part);
}

/* Collision probability of eq. (yoso-expectation) for a cosine similarity x. */
double oracle_collision_prob(double x, int tau)
{
    if (x > 1.0) x = 1.0;
    if (x < -1.0) x = -1.0;
    return pow(1.0 - acos(x) / M_PI, tau);
}

/* Exact expectation over hash functions (YOSO-E), O(n^2 d):
 *   P_ij = (1 - arccos(cos(q_i, k_j))/pi)^tau
 *   ey  = P v,  edv = P^T dy,
 *   edq = (tau/2) [(dy v^T) .* P] k,  edk = (tau/2) [(dy v^T) .* P]^T q,
 *   tdq (optional) = [(dy v^T) .* tau P^{(tau-1)/tau} ./ (pi sqrt(1 - cos^2))] k,
 *   the true gradient of eq. (gradient-q) for unit rows (diverges as cos -> 1),
 *   and tdk (optional) = [...]^T q, its counterpart for K.  With floor > 0 the
 *   factor 1 - cos^2 is raised to at least `floor` (the bound *YOSO's estimator
 *   uses; 0 leaves it unbounded).
 * The cosine is taken of the rows as given, normalised by their norms. */
void oracle_expectation(const double *q, const double *k, const double *v, const double *dy,
                        int64_t bh, int64_t nq, int64_t nk, int d, int tau, double floor_,
                        double *ey, double *edv, double *edq, double *edk, double *tdq, double *tdk)
{
    memset(ey, 0, sizeof(double) * bh * nq * d);
    memset(edv, 0, sizeof(double) * bh * nk * d);
    memset(edq, 0, sizeof(double) * bh * nq * d);
    memset(edk, 0, sizeof(double) * bh * nk * d);
    if (tdq) memset(tdq, 0, sizeof(double) * bh * nq * d);
    if (tdk) memset(tdk, 0, sizeof(double) * bh * nk * d);
    for (int64_t b = 0; b < bh; b++) {
        const double *qb = q + b * nq * d, *kb = k + b * nk * d;
        const double *vb = v + b * nk * d, *dyb = dy + b * nq * d;
        for (int64_t i = 0; i < nq; i++) {
            for (int64_t j = 0; j < nk; j++) {
                double dot = 0.0, nqi = 0.0, nkj = 0.0, g = 0.0;
                for (int l = 0; l < d; l++) {
                    dot += qb[i * d + l] * kb[j * d + l];
                    nqi += qb[i * d + l] * qb[i * d + l];
                    nkj += kb[j * d + l] * kb[j * d + l];
                    g += dyb[i * d + l] * vb[j * d + l];
                }
                double cosv = dot / sqrt(nqi * nkj);
                if (cosv > 1.0) cosv = 1.0;
                if (cosv < -1.0) cosv = -1.0;
                const double p = pow(1.0 - acos(cosv) / M_PI, tau);
                for (int l = 0; l < d; l++) {
                    ey[(b * nq + i) * d + l] += p * vb[j * d + l];
                    edv[(b * nk + j) * d + l] += p * dyb[i * d + l];
                    edq[(b * nq + i) * d + l] += (tau / 2.0) * g * p * kb[j * d + l];
                    edk[(b * nk + j) * d + l] += (tau / 2.0) * g * p * qb[i * d + l];
                }
                if (tdq || tdk) {
                    double r = 1.0 - cosv * cosv;
                    if (r < floor_) r = floor_;
                    const double w = tau * pow(1.0 - acos(cosv) / M_PI, tau - 1) / (M_PI * sqrt(r));
                    for (int l = 0; l < d; l++) {
                        if (tdq) tdq[(b * nq + i) * d + l] += g * w * kb[j * d + l];
                        if (tdk) tdk[(b * nk + j) * d + l] += g * w * qb[i * d + l];
                    }
                }
            }
        }
    }
}

/* Row l2 normalisation: y[r] = x[r] / ||x[r]|| (the zero row stays zero).
 * x, y: [rows][d]. */
void oracle_l2_normalize(const double *x, int64_t rows, int d, double *y)
{
    for (int64_t r = 0; r < rows; r++) {
        double ss = 0.0;
        for (int l = 0; l < d; l++) ss += x[r * d + l] * x[r * d + l];
        const double nrm = sqrt(ss);
        for (int l = 0; l < d; l++) y[r * d + l] = nrm > 0.0 ? x[r * d + l] / nrm : 0.0;
    }
}

/* Backward of the map above: dx[r][j] = sum_i dy[r][i] * dy_i/dx_j, with the
 * Jacobian of y = x/||x|| written out entry by entry,
 *   dy_i/dx_j = delta_ij / ||x|| - x_i x_j / ||x||^3,
 * and 0 for the zero row.  x (the forward's input), dy, dx: [rows][d]. */
void oracle_l2_normalize_backward(const double *x, const double *dy, int64_t rows, int d, double *dx)
{
    for (int64_t r = 0; r < rows; r++) {
        const double *xr = x + r * d, *gr = dy + r * d;
        double ss = 0.0;
        for (int l = 0; l < d; l++) ss += xr[l] * xr[l];
        const double nrm = sqrt(ss);
        for (int j = 0; j < d; j++) {
            double acc = 0.0;
            if (nrm > 0.0) {
                for (int i = 0; i < d; i++) {
                    const double jac = (i == j ? 1.0 / nrm : 0.0) - xr[i] * xr[j] / (nrm * nrm * nrm);
                    acc += gr[i] * jac;
                }
            }
            dx[r * d + j] = acc;
        }
    }
}

/* Sylvester's Walsh-Hadamard matrix of order d (a power of two), built by the
 * doubling H_1 = [1], H_2k = [[H_k, H_k], [H_k, -H_k]].  H: d*d row-major. */
void oracle_hadamard(int d, double *H)
{
    H[0] = 1.0;
    for (int k = 1; k < d; k *= 2) {
        /* the k x k block in the top-left corner is H_k; fill the other three */
        for (int i = 0; i < k; i++) {
            for (int j = 0; j < k; j++) {
                const double h = H[i * d + j];
                H[i * d + j + k] = h;
                H[(i + k) * d + j] = h;
                H[(i + k) * d + j + k] = -h;
            }
        }
    }
}

/* Hyperplanes of the fast hash (Sec. 3.2 "Speed-up"; the pseudo-random rotation of
 * Andoni et al. 2015): for rotation r = 0 .. ceil(m*tau/d) - 1
 *   M_r = (1/d) H D3 H D2 H D1,   D_i = diag(+-1 from signs[3r + i - 1]),
 * and column c = r*d + l of R (c < m*tau) is row l of M_r:  R[j][c] = M_r[l][j].
 * d is a power of two, at most 64.  R: d x (m*tau) row-major. */
void oracle_fast_hyperplanes(const uint64_t *signs, int d, int m, int tau, double *R)
{
    const int ncol = m * tau;
    const int nrot = (ncol + d - 1) / d;
    double *H = malloc(sizeof(double) * d * d);
    double *M = malloc(sizeof(double) * d * d);
    double *T = malloc(sizeof(double) * d * d);
    oracle_hadamard(d, H);
    for (int r = 0; r < nrot; r++) {
        /* M = I; then, for D1, D2, D3 in turn, M <- H D M */
        for (int i = 0; i < d * d; i++) M[i] = 0.0;
        for (int i = 0; i < d; i++) M[i * d + i] = 1.0;
        for (int round = 0; round < 3; round++) {
            const uint64_t s = signs[3 * r + round];
            for (int i = 0; i < d; i++)          /* T = D M */
                for (int j = 0; j < d; j++)
                    T[i * d + j] = ((s >> i) & 1u) ? -M[i * d + j] : M[i * d + j];
            for (int i = 0; i < d; i++)          /* M = H T */
                for (int j = 0; j < d; j++) {
                    double acc = 0.0;
                    for (int k = 0; k < d; k++) acc += H[i * d + k] * T[k * d + j];
                    M[i * d + j] = acc;
                }
        }
        for (int l = 0; l < d; l++) {
            const int c = r * d + l;
            if (c >= ncol) break;
            for (int j = 0; j < d; j++) R[(int64_t)j * ncol + c] = M[l * d + j] / d;
        }
    }
    free(H); free(M); free(T);
}
