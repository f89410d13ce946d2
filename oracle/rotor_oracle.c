/*
 * Oracle for the optimal persistent checkpointing dynamic program of
 * Beaumont, Eyraud-Dubois, Hermann, Joly, Shilova, "Optimal checkpointing for
 * heterogeneous chains: how to train deep neural networks with limited
 * memory" (arXiv 1911.13214).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, single-threaded
 * restatement of the paper's recurrence used to check the GPU library.  Only
 * the test suite, the smoke check and the CPU-baseline leg of the benchmark
 * may load it.  It shares no code, header or table with the GPU library.
 *
 * Integers everywhere: times and sizes are integer units (memory already
 * discretised into slots, Section 5.2), costs are int64 and infinity is
 * INT64_MAX.
 *
 * Inputs: a packed int64 array p[6][L] with rows u_f, u_b, omega_a,
 * omega_abar, o_f, o_b; stage l (1-based, as in Section 3.1) is column l-1.
 * omega_delta is taken equal to omega_a (the paper states they are equal in
 * practice, Section 3.1).
 *
 * Readings of the paper used here (each also listed in the design notes):
 *  - Algorithm 1 fills C by (s, t) with s outer; C(s,t,.) needs C(s',t,.) for
 *    s' > s, so the table is filled by increasing t - s instead.  Every term
 *    of Theorem 1 is a strictly shorter sub-chain.
 *  - The library's L counts every stage it is given (the loss, if modelled,
 *    is simply the last stage), and budgets m run over 0..M with the chain
 *    input a^{s-1} not counted, as in the definition of C_BP (Section 4.2).
 *  - A shifted budget m - omega < 0 is infeasible.
 *  - Among the C_1 candidates the smallest s' wins ties, and C_1 wins ties
 *    against C_2.  The decision table holds s' (>= s+1) for a C_1 choice,
 *    0 for C_2 or the leaf rule, -1 for an infeasible cell.
 *  - Algorithm 2 emits F_none up to stage s'-1 (the C_ck cost charges
 *    u_f^s .. u_f^{s'-1}, and a^{s'-1} is the next stored value).
 *
 * Parity is pinned outside this file: brute force over all persistent
 * schedules with an independent memory/time simulator, closed forms for the
 * homogeneous chain, the all-F_all closed form, monotonicity, the
 * feasibility threshold recurrence and replay of reconstructed sequences.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_INF INT64_MAX

enum { R_UF = 0, R_UB, R_WA, R_WAB, R_OF, R_OB };
enum { OP_F_CK = 0, OP_F_NONE = 1, OP_F_ALL = 2, OP_B = 3 };

typedef struct {
    int L;
    int64_t M;
    const int64_t *p; /* [6][L] */
} orc_chain;

static int64_t par(const orc_chain *c, int row, int l) { return c->p[(int64_t)row * c->L + (l - 1)]; }
static int64_t uf(const orc_chain *c, int l) { return par(c, R_UF, l); }
static int64_t ub(const orc_chain *c, int l) { return par(c, R_UB, l); }
static int64_t wa(const orc_chain *c, int l) { return par(c, R_WA, l); }
static int64_t wd(const orc_chain *c, int l) { return par(c, R_WA, l); } /* omega_delta = omega_a */
static int64_t wab(const orc_chain *c, int l) { return par(c, R_WAB, l); }
static int64_t of(const orc_chain *c, int l) { return par(c, R_OF, l); }
static int64_t ob(const orc_chain *c, int l) { return par(c, R_OB, l); }

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

/* Row of the pair (s,t), 1 <= s <= t <= L, in the oracle's own storage:
 * the upper triangle stored s-major (row s holds t = s..L). */
int64_t oracle_row(int L, int s, int t)
{
    return (int64_t)(s - 1) * (L + 1) - (int64_t)(s - 1) * s / 2 + (t - s);
}

/* m_all(s,t), Section 4.2: the larger of the peak of F_all^s with delta^t
 * stored and the peak of B^s with delta^s stored. */
int64_t oracle_m_all(int L, const int64_t *p, int s, int t)
{
    orc_chain c = {L, 0, p};
    return max64(wd(&c, t) + wab(&c, s) + of(&c, s), wd(&c, s) + wab(&c, s) + ob(&c, s));
}

/* m_none(s,t), s < t, Section 4.2: the peak of F_ck^s followed by
 * F_none^{s+1..t-1} with delta^t stored.  The inner max over j is empty when
 * t = s + 1. */
int64_t oracle_m_none(int L, const int64_t *p, int s, int t)
{
    orc_chain c = {L, 0, p};
    int64_t g = wd(&c, t) + wa(&c, s) + of(&c, s);
    for (int j = s + 1; j < t; ++j)
        g = max64(g, wd(&c, t) + wa(&c, j - 1) + wa(&c, j) + of(&c, j));
    return g;
}

/* The oracle's own input domain: what its int64 arithmetic handles without
 * overflow, whatever any other implementation supports.
 *  - 1 <= L <= 32767 (decisions are int16) and 0 <= M < 2^31;
 *  - every value >= 0;
 *  - sizes and overheads below 2^60: a gate adds at most four of them;
 *  - L * sum(u_f) + sum(u_b) below 2^62.  A C_1 or C_2 candidate of the pair
 *    (s, t) is the time of a persistent schedule of [s, t] (Theorem 1), in
 *    which no stage runs forward more than t - s + 1 <= L times, so every
 *    candidate and every partial sum of one stays below 2^62 < INT64_MAX.
 * Theorem 1 defines C for any non-negative integers; these limits only keep
 * the arithmetic exact. */
int oracle_check(int L, int64_t M, const int64_t *p)
{
    const uint64_t cost_bound = (uint64_t)1 << 62;
    if (L < 1 || L > 32767 || M < 0 || M >= ((int64_t)1 << 31))
        return -1;
    orc_chain c = {L, M, p};
    uint64_t suf = 0, sub = 0;
    for (int l = 1; l <= L; ++l) {
        if (uf(&c, l) < 0 || ub(&c, l) < 0 || (uint64_t)uf(&c, l) >= cost_bound ||
            (uint64_t)ub(&c, l) >= cost_bound)
            return -1;
        int64_t s[4] = {wa(&c, l), wab(&c, l), of(&c, l), ob(&c, l)};
        for (int k = 0; k < 4; ++k)
            if (s[k] < 0 || s[k] >= ((int64_t)1 << 60))
                return -1;
        suf += (uint64_t)uf(&c, l);
        sub += (uint64_t)ub(&c, l);
        if (suf >= cost_bound || sub >= cost_bound)
            return -1;
    }
    /* L * suf + sub < 2^62, written without overflow */
    if (suf > (cost_bound - sub) / (uint64_t)L)
        return -1;
    return 0;
}

/* Theorem 1 for a single cell (s,t,m), evaluated from the table C that
 * already holds every strictly shorter sub-chain.  Candidates are taken in
 * increasing s' with a strict <, then C_2 with a strict <.  Writes the
 * decision to *dec. */
int64_t oracle_cell(int L, int64_t M, const int64_t *p, const int64_t *C, int s, int t, int64_t m, int16_t *dec)
{
    orc_chain c = {L, M, p};
    const int64_t W = M + 1;
    int64_t best = ORC_INF;
    int arg = -1;
    if (s == t) { /* Eq. (DP:Init) */
        if (m >= oracle_m_all(L, p, s, s)) {
            best = uf(&c, s) + ub(&c, s);
            arg = 0;
        }
        *dec = (int16_t)arg;
        return best;
    }
    if (m >= oracle_m_none(L, p, s, t)) { /* C_1 = min over s' of C_ck */
        int64_t sum = 0; /* sum of u_f^k for k = s .. s'-1 */
        for (int sp = s + 1; sp <= t; ++sp) {
            sum += uf(&c, sp - 1);
            int64_t r = m - wa(&c, sp - 1);
            if (r < 0)
                continue;
            int64_t A = C[oracle_row(L, sp, t) * W + r];
            int64_t B = C[oracle_row(L, s, sp - 1) * W + m];
            if (A == ORC_INF || B == ORC_INF)
                continue;
            int64_t v = sum + A + B;
            if (v < best) {
                best = v;
                arg = sp;
            }
        }
    }
    if (m >= oracle_m_all(L, p, s, t)) { /* C_2 = C_all */
        int64_t r = m - wab(&c, s);
        if (r >= 0) {
            int64_t A = C[oracle_row(L, s + 1, t) * W + r];
            if (A != ORC_INF) {
                int64_t v = uf(&c, s) + A + ub(&c, s);
                if (v < best) {
                    best = v;
                    arg = 0;
                }
            }
        }
    }
    *dec = (int16_t)arg;
    return best;
}

/* Fill the whole table (Theorem 1) by increasing sub-chain length d = t - s.
 * C has L(L+1)/2 rows of M+1 costs, D the matching decisions, both in the
 * oracle_row order.  Returns 0, or -1 if the input is outside the domain.
 *
 * For each cell the budgets m are independent of one another, so the C_1
 * candidates are swept one s' at a time over all m (two whole rows at once)
 * instead of one m at a time; for every fixed m the candidates are still met
 * in increasing s' under a strict <, then C_2 under a strict <, which is
 * exactly the order of oracle_cell. */
int oracle_solve(int L, int64_t M, const int64_t *p, int64_t *C, int16_t *D)
{
    if (oracle_check(L, M, p))
        return -1;
    orc_chain c = {L, M, p};
    const int64_t W = M + 1;

    for (int s = 1; s <= L; ++s) { /* Eq. (DP:Init) */
        int64_t *row = C + oracle_row(L, s, s) * W;
        int16_t *drow = D + oracle_row(L, s, s) * W;
        int64_t g = oracle_m_all(L, p, s, s);
        for (int64_t m = 0; m <= M; ++m) {
            row[m] = m >= g ? uf(&c, s) + ub(&c, s) : ORC_INF;
            drow[m] = m >= g ? 0 : -1;
        }
    }

    for (int d = 1; d < L; ++d) {
        for (int s = 1; s + d <= L; ++s) {
            int t = s + d;
            int64_t *best = C + oracle_row(L, s, t) * W;
            int16_t *arg = D + oracle_row(L, s, t) * W;
            for (int64_t m = 0; m <= M; ++m) {
                best[m] = ORC_INF;
                arg[m] = -1;
            }
            /* C_1, gated by m >= m_none(s,t) */
            int64_t g1 = oracle_m_none(L, p, s, t);
            int64_t sum = 0;
            for (int sp = s + 1; sp <= t; ++sp) {
                sum += uf(&c, sp - 1);
                int64_t w = wa(&c, sp - 1);
                const int64_t *right = C + oracle_row(L, sp, t) * W; /* C(s', t, .) */
                const int64_t *left = C + oracle_row(L, s, sp - 1) * W; /* C(s, s'-1, .) */
                for (int64_t m = max64(g1, w); m <= M; ++m) {
                    int64_t A = right[m - w], B = left[m];
                    if (A == ORC_INF || B == ORC_INF)
                        continue;
                    int64_t v = sum + A + B;
                    if (v < best[m]) {
                        best[m] = v;
                        arg[m] = (int16_t)sp;
                    }
                }
            }
            /* C_2, gated by m >= m_all(s,t) */
            int64_t g2 = oracle_m_all(L, p, s, t);
            int64_t w = wab(&c, s);
            const int64_t *below = C + oracle_row(L, s + 1, t) * W; /* C(s+1, t, .) */
            for (int64_t m = max64(g2, w); m <= M; ++m) {
                int64_t A = below[m - w];
                if (A == ORC_INF)
                    continue;
                int64_t v = uf(&c, s) + A + ub(&c, s);
                if (v < best[m]) {
                    best[m] = v;
                    arg[m] = 0;
                }
            }
        }
    }
    return 0;
}

/* Algorithm 2 (OptRec): rebuild the sequence from the cost table alone, by
 * finding which option of Theorem 1 attains C(s,t,m).  The smallest s' whose
 * C_ck equals the cell is taken, and C_1 is preferred to C_2, matching the
 * tie rule of the fill.  Appends to ops[2*k] = kind, ops[2*k+1] = stage. */
typedef struct {
    orc_chain c;
    const int64_t *C;
    int32_t *ops;
    int64_t cap, n;
    int err;
} orc_rec;

static void emit(orc_rec *r, int kind, int stage)
{
    if (r->n < r->cap) {
        r->ops[2 * r->n] = kind;
        r->ops[2 * r->n + 1] = stage;
    }
    r->n++;
}

static void opt_rec(orc_rec *r, int s, int t, int64_t m)
{
    const orc_chain *c = &r->c;
    const int L = c->L;
    const int64_t W = c->M + 1;
    if (m < 0 || r->C[oracle_row(L, s, t) * W + m] == ORC_INF) {
        r->err = 1; /* infeasible */
        return;
    }
    int64_t cst = r->C[oracle_row(L, s, t) * W + m];
    if (s == t) {
        emit(r, OP_F_ALL, s);
        emit(r, OP_B, s);
        return;
    }
    if (m >= oracle_m_none(L, c->p, s, t)) {
        int64_t sum = 0;
        for (int sp = s + 1; sp <= t; ++sp) {
            sum += uf(c, sp - 1);
            int64_t rr = m - wa(c, sp - 1);
            if (rr < 0)
                continue;
            int64_t A = r->C[oracle_row(L, sp, t) * W + rr];
            int64_t B = r->C[oracle_row(L, s, sp - 1) * W + m];
            if (A == ORC_INF || B == ORC_INF || sum + A + B != cst)
                continue;
            emit(r, OP_F_CK, s);
            for (int k = s + 1; k <= sp - 1; ++k)
                emit(r, OP_F_NONE, k);
            opt_rec(r, sp, t, rr);
            opt_rec(r, s, sp - 1, m);
            return;
        }
    }
    emit(r, OP_F_ALL, s);
    opt_rec(r, s + 1, t, m - wab(c, s));
    emit(r, OP_B, s);
}

/* Sequence for the whole chain [1, L] at budget m.  ops holds cap pairs of
 * int32 (kind, stage).  Returns the number of operations (which may exceed
 * cap: only the first cap are written), or -1 if C(1,L,m) is infinite, -2 on
 * bad arguments. */
int64_t oracle_reconstruct(int L, int64_t M, const int64_t *p, const int64_t *C, int64_t m, int32_t *ops, int64_t cap)
{
    if (m < 0 || m > M || L < 1)
        return -2;
    orc_rec r = {{L, M, p}, C, ops, cap, 0, 0};
    opt_rec(&r, 1, L, m);
    return r.err ? -1 : r.n;
}

/* ---- front end: discretisation and the store-everything memory ----------- */

/* Section 5.2: with a memory limit mem and S slots of mem / S each, a size v
 * takes the smallest whole number of slots q with q * (mem / S) >= v, that
 * is q * mem >= v * S. */
int64_t oracle_slots(int64_t v, int64_t mem, int64_t S)
{
    const unsigned __int128 need = (unsigned __int128)v * (unsigned __int128)S;
    unsigned __int128 q = need / (unsigned __int128)mem;
    if (q * (unsigned __int128)mem < need)
        q += 1;
    return (int64_t)q;
}

/* p_out[6][L] = p_in with the four size rows (omega_a, omega_abar, o_f, o_b)
 * in slots; the time rows are copied. */
void oracle_discretize(int L, const int64_t *p_in, int64_t mem, int64_t S, int64_t *p_out)
{
    for (int row = 0; row < 6; ++row)
        for (int l = 0; l < L; ++l) {
            const int64_t v = p_in[(int64_t)row * L + l];
            const int size_row = row == R_WA || row == R_WAB || row == R_OF || row == R_OB;
            p_out[(int64_t)row * L + l] = size_row ? oracle_slots(v, mem, S) : v;
        }
}

/* Peak memory of F_all^1 .. F_all^L, B^L .. B^1, replayed with the
 * accounting of Theorem 1: the chain input a^0 is not counted, delta^L is
 * stored from the start, an operation's peak is what is stored plus its
 * output and overhead, and B^j's output delta^{j-1} is not counted while B^j
 * runs (the m_all backward term). */
int64_t oracle_store_all_peak(int L, const int64_t *p)
{
    orc_chain ch = {L, 0, p};
    int64_t stored = wd(&ch, L); /* delta^L */
    int64_t peak = 0;
    for (int j = 1; j <= L; ++j) {
        /* F_all^j reads a^{j-1} (inside abar^{j-1}, or a^0) and writes abar^j */
        peak = max64(peak, stored + wab(&ch, j) + of(&ch, j));
        stored += wab(&ch, j);
    }
    for (int j = L; j >= 1; --j) {
        /* B^j reads delta^j and abar^j, both stored */
        peak = max64(peak, stored + ob(&ch, j));
        /* then abar^j and delta^j are freed and delta^{j-1} is stored */
        stored -= wab(&ch, j) + wd(&ch, j);
        if (j > 1)
            stored += wd(&ch, j - 1);
    }
    return peak;
}
