/*
 * rotor.h -- C ABI of the MI355X (gfx950) solver for optimal persistent
 * activation checkpointing on heterogeneous chains.
 *
 * The method is the dynamic program of Beaumont, Eyraud-Dubois, Hermann,
 * Joly and Shilova, "Optimal checkpointing for heterogeneous chains"
 * (arXiv 1911.13214): Theorem 1 (Section 4.2) defines the optimal time
 * C_BP(s, t, m) of the sub-chain [s, t] under a memory budget m, Algorithm 1
 * fills the table and Algorithm 2 rebuilds the operation sequence.
 *
 * Units.  Times and sizes are integers: the caller has already expressed
 * memory as a number of slots (Section 5.2 discretises sizes into S slots,
 * rounded up).  Costs are int64; an infeasible cell holds ROTOR_INF.
 *
 * Chain parameters.  A chain of L stages (stages are numbered 1..L as in
 * Section 3.1; the loss, if modelled, is simply the last stage) is described
 * by six rows of L int64 values -- the model inputs of Section 5.1 and
 * Table 1:
 *   ROTOR_ROW_UF    u_f^l   time of any forward operation of stage l
 *   ROTOR_ROW_UB    u_b^l   time of the backward operation B^l
 *   ROTOR_ROW_WA    w_a^l   size of the stage output a^l; also the size of
 *                           the gradient delta^l (the paper takes them equal)
 *   ROTOR_ROW_WABAR w_abar^l size of abar^l, all data F_all^l keeps for B^l
 *   ROTOR_ROW_OF    o_f^l   memory overhead of the forward operations
 *   ROTOR_ROW_OB    o_b^l   memory overhead of B^l
 * Stage l sits at column l-1.  A batch of n_chains chains of equal L is
 * packed chain-major: params[c][row][l-1], c = 0..n_chains-1.
 *
 * Domain.  Every value is >= 0; sizes and overheads are < 2^30; M < 2^28;
 * for every chain L * sum(u_f) + sum(u_b) < 2^44 (this bounds every finite
 * cost: a persistent schedule runs each forward at most L times).  These are
 * limits of this library's number formats, narrower than the problem itself.
 * rotor_check_params verifies them on a host copy; rotor_solve also checks
 * every chain on the device and records the result in its workspace, which
 * rotor_solve_status reports, and rotor_reconstruct refuses a chain outside
 * the domain.  The kernels read and write only within the caller's buffers
 * whatever the parameter values (every shifted budget is checked to lie in
 * [0, m] before it is read); outside the domain the table contents are
 * unspecified.
 *
 * Budgets.  Column m = 0..M of the tables is the budget of the definition of
 * C_BP: the input a^{s-1} of the sub-chain is not counted, the gradient
 * delta^t is.  To count the chain input a^0 as Algorithm 1 does, query the
 * row (1, L) at M - size(a^0).
 *
 * Table layout (device memory, caller-owned).  Per chain, the L(L+1)/2 pairs
 * (s, t), 1 <= s <= t <= L, are stored s-major (by s, then t):
 *   row(s, t) = (s-1)*L - (s-1)*(s-2)/2 + (t-s)
 * Each row holds `pitch` elements, pitch = M+1 rounded up to a multiple of
 * 32 (256 bytes of costs); only columns 0..M are written.  The cost table is
 * int64 and the decision table int16, with the same indexing:
 *   element(c, s, t, m) = (c * rows + row(s, t)) * pitch + m,
 *   rows = L(L+1)/2.
 * Decision values: -1 infeasible; 0 the sequence starts with F_all^s (the C_2
 * option of Theorem 1, or the single-stage rule of Eq. (DP:Init)); s' in
 * [s+1, t] it starts with F_ck^s and stores a^{s'-1} next (option C_1 with
 * split s').  Among equal costs the smallest s' is chosen, and C_1 is
 * preferred to C_2, so the table is unique.
 *
 * Streams.  `stream` is a hipStream_t passed as void* (NULL: the default
 * stream).  Entry points that take device buffers only enqueue work and
 * return; argument errors are reported synchronously by the return value,
 * device-side failures surface at the caller's next synchronisation.  Before
 * enqueuing, they clear the calling thread's pending HIP error (the one
 * hipGetLastError would return), so that ROTOR_EDEVICE reports a failure of
 * their own launches only.  The
 * library allocates no device memory (the caller passes the solve's
 * workspace) and keeps no state between calls but two: the static workspace
 * of rotor_solve_noalloc, one device array per device; and, for the blocked
 * fill, one side stream and two events per device (created by the first
 * solve on the device, kept until the process ends), on which part of each
 * middle product runs beside the edge rounds before it (edges by
 * anti-diagonal rounds, not by rows) and which the solve joins
 * back into `stream` before it returns (if the side stream cannot be
 * created, every launch goes to `stream`).  Solves hold a lock while they
 * enqueue; concurrent calls on distinct output buffers and workspaces are
 * independent.
 */
#ifndef ROTOR_H
#define ROTOR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#ifndef ROTOR_API
#define ROTOR_API __attribute__((visibility("default")))
#endif

#define ROTOR_VERSION 1
#define ROTOR_INF INT64_MAX

/* Status codes. */
#define ROTOR_OK 0
#define ROTOR_EINVAL (-1)       /* bad argument (null pointer, size out of range) */
#define ROTOR_EDOMAIN (-2)      /* a parameter value is outside the domain above */
#define ROTOR_EDEVICE (-3)      /* the HIP runtime refused a launch or query */
#define ROTOR_INFEASIBLE (-4)   /* no sequence fits the budget: C(1, L, m) is infinite */
#define ROTOR_ECAPACITY (-5)    /* the output array is too small; the count holds the size needed */
#define ROTOR_ECORRUPT (-6)     /* the decision table is not one this library wrote */
#define ROTOR_ESEQUENCE (-7)    /* an operation sequence is not valid (rotor_sequence_cost) */

/* Rows of the packed parameter array. */
#define ROTOR_ROW_UF 0
#define ROTOR_ROW_UB 1
#define ROTOR_ROW_WA 2
#define ROTOR_ROW_WABAR 3
#define ROTOR_ROW_OF 4
#define ROTOR_ROW_OB 5
#define ROTOR_N_ROWS 6

/* Operations of Table 1. */
#define ROTOR_F_CK 0   /* forward, keep the input a^{l-1} (checkpoint) */
#define ROTOR_F_NONE 1 /* forward, keep nothing but the output a^l */
#define ROTOR_F_ALL 2  /* forward, keep abar^l for the backward */
#define ROTOR_B 3      /* backward B^l */

typedef struct {
    int32_t kind;  /* ROTOR_F_CK, ROTOR_F_NONE, ROTOR_F_ALL or ROTOR_B */
    int32_t stage; /* 1..L */
} rotor_op;

/* Largest L accepted by rotor_solve (decisions are int16) and by
 * rotor_reconstruct (its walk keeps one 8-byte frame per pending sub-chain in
 * 64 KiB of LDS). */
#define ROTOR_MAX_L 32767
#define ROTOR_MAX_L_RECONSTRUCT 8191
#define ROTOR_MAX_CHAINS 65535

/* Library version (ROTOR_VERSION). */
ROTOR_API int32_t rotor_version(void);

/* Short English text for a status code. */
ROTOR_API const char *rotor_status_string(int32_t status);

/* Table geometry for n_chains chains of L stages and budgets 0..M (layout
 * above).  Any output pointer may be NULL.  Host only; no device work.
 * Returns ROTOR_OK, or ROTOR_EINVAL if n_chains, L or M is out of range or a
 * byte count would overflow 64 bits. */
ROTOR_API int32_t rotor_layout(int32_t n_chains, int32_t L, int64_t M, int64_t *pitch, int64_t *rows_per_chain,
                     uint64_t *cost_bytes, uint64_t *dec_bytes);

/* Row of the pair (s, t) within one chain (layout above), or -1 unless
 * 1 <= s <= t <= L.  Host only. */
ROTOR_API int64_t rotor_row_index(int32_t L, int32_t s, int32_t t);

/* Check HOST parameters [n_chains][6][L] against the domain above.
 * Returns ROTOR_OK, ROTOR_EINVAL (null pointer, sizes out of range) or
 * ROTOR_EDOMAIN (a value out of range).  Host only. */
ROTOR_API int32_t rotor_check_params(const int64_t *h_params, int32_t n_chains, int32_t L, int64_t M);

/* Bytes of device workspace rotor_solve needs for these sizes: per-pair
 * gates and saturation budgets, prefix sums, a few words per block of 16
 * stages, a domain status
 * word per chain, a compact 4-byte-per-cell copy of the cost table (about
 * 40% of cost_bytes + dec_bytes) and, for chains of more than 16 stages, a
 * 2-byte copy of the cells of the 16 x 16 diagonal blocks.  Host only.
 * Returns ROTOR_OK or ROTOR_EINVAL (as rotor_layout). */
ROTOR_API int32_t rotor_workspace_bytes(int32_t n_chains, int32_t L, int64_t M, uint64_t *bytes);

/* Fill the cost table C_BP(s, t, m) and the decision table for every chain,
 * every pair 1 <= s <= t <= L and every budget 0 <= m <= M: Theorem 1,
 * Eq. (DP:Init) for t = s and Eq. (DP:mainrec) for t > s, evaluated so that
 * every term is read after it is final (Algorithm 1's printed loop order does
 * not respect this; the fill goes by increasing t - s within 16 x 16 blocks of
 * pairs, block-diagonal by block-diagonal).
 *
 *   d_params  DEVICE, read only: [n_chains][6][L] int64 (layout above).
 *   d_cost    DEVICE, written: int64, rotor_layout's cost_bytes.
 *   d_dec     DEVICE, written: int16, rotor_layout's dec_bytes.
 *   d_work    DEVICE scratch of at least rotor_workspace_bytes, caller-owned;
 *             its contents on entry do not matter and on exit are unspecified.
 *   stream    hipStream_t or NULL.
 * Asynchronous.  Returns ROTOR_OK once every kernel is enqueued, ROTOR_EINVAL
 * for a null or misaligned pointer, a size out of range or a workspace too
 * small, ROTOR_EDEVICE if a launch fails.  Allocates nothing.  Calls that
 * share a workspace must not overlap. */
ROTOR_API int32_t rotor_solve(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost,
                              int16_t *d_dec, void *d_work, uint64_t work_bytes, void *stream);

/* Workspace bytes of rotor_solve_noalloc: a static device array of this size
 * (128 MiB), held by every device the library runs on until the process
 * ends. */
#define ROTOR_NOALLOC_WORK_BYTES (128ull << 20)

/* rotor_solve for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same fill and tables, with the workspace taken from a static device
 * array of ROTOR_NOALLOC_WORK_BYTES bytes per device instead of a caller
 * buffer, and every launch on `stream` (no side stream: the blocked fill's
 * middle products wait for the edges before them).  The caller still passes parameters and tables (as for
 * rotor_solve).  It calls no hipMalloc, hipFree or allocating library
 * routine.  Every call on one device shares that device's array, so calls
 * that overlap on one device (different streams, or host threads) race and
 * must be serialised by the caller; nothing left in the array by an earlier
 * call affects a later one.  The per-device domain status is not kept for
 * rotor_solve_status (use rotor_check_params on the host).
 * Returns ROTOR_OK once every kernel is enqueued, ROTOR_EINVAL for a null or
 * misaligned pointer or a size out of range, ROTOR_ECAPACITY if the
 * workspace these sizes need (rotor_workspace_bytes) exceeds
 * ROTOR_NOALLOC_WORK_BYTES, ROTOR_EDEVICE if the array's address cannot be
 * found or a launch fails. */
ROTOR_API int32_t rotor_solve_noalloc(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M,
                                      int64_t *d_cost, int16_t *d_dec, void *stream);

/* Domain report of the solve that last used this workspace: waits for
 * `stream` (the stream of that solve), then reads the status word the fill
 * recorded for each chain.
 *   d_work, work_bytes  DEVICE: the workspace given to rotor_solve (same
 *                       n_chains, L, M).
 *   h_chain_status      HOST, n_chains int32 written (may be NULL):
 *                       ROTOR_OK, or ROTOR_EDOMAIN for a chain whose
 *                       parameters are outside the domain (its tables are
 *                       unspecified).
 * Returns ROTOR_OK if every chain was in the domain, ROTOR_EDOMAIN if one
 * was not, ROTOR_EINVAL for bad arguments or a workspace no solve has
 * written, ROTOR_EDEVICE if the copy fails.  Synchronous; allocates no device
 * memory. */
ROTOR_API int32_t rotor_solve_status(const void *d_work, uint64_t work_bytes, int32_t n_chains, int32_t L, int64_t M,
                                     int32_t *h_chain_status, void *stream);

/* Fill orders of rotor_solve_schedule.  All fill the same tables, bit for
 * bit; they differ in speed.
 *   ROTOR_SCHEDULE_BLOCKED   16 x 16 blocks of pairs: register-tiled min-plus
 *                            products for the splits that reach across
 *                            blocks; the splits inside the block's own rows
 *                            and columns ("edges") by rows (16 launches per
 *                            block-diagonal) when a block-diagonal holds at
 *                            least 256 blocks over all chains, else by
 *                            anti-diagonals (30 short launches); the fast
 *                            order for large tables.
 *   ROTOR_SCHEDULE_DIAGONAL  one launch per t - s over all pairs (the
 *                            wavefront the recurrence allows), the splits of
 *                            a pair spread over four waves from t - s = 16 on;
 *                            fewer launches, the fast order for small tables.
 *   ROTOR_SCHEDULE_AUTO      DIAGONAL when the table has at most 2e9 split
 *                            candidates (L^3/6 (M+1)) for one chain, or 4e8
 *                            summed over a batch, or when one chain has
 *                            M < 63; BLOCKED otherwise (the order rotor_solve
 *                            uses).
 *   ROTOR_SCHEDULE_BLOCKED_ROWS, ROTOR_SCHEDULE_BLOCKED_ROUNDS
 *                            BLOCKED with the edges of every block-diagonal
 *                            by rows, or by anti-diagonals.
 *   ROTOR_SCHEDULE_BLOCKED_SERIAL
 *                            BLOCKED with every middle product on the
 *                            caller's stream after the edges of the
 *                            block-diagonal before it.  The other blocked
 *                            orders run the splits of a middle product that
 *                            reach no further than two block-diagonals back
 *                            on a second stream of the library's (one per
 *                            device, created by the first solve on the
 *                            device and kept until the process ends) beside
 *                            those edges, and join it before the product's
 *                            remaining splits. */
#define ROTOR_SCHEDULE_AUTO 0
#define ROTOR_SCHEDULE_BLOCKED 1
#define ROTOR_SCHEDULE_DIAGONAL 2
#define ROTOR_SCHEDULE_BLOCKED_ROWS 3
#define ROTOR_SCHEDULE_BLOCKED_ROUNDS 4
#define ROTOR_SCHEDULE_BLOCKED_SERIAL 5

/* rotor_solve with an explicit fill order; ROTOR_EINVAL for an unknown one. */
ROTOR_API int32_t rotor_solve_schedule(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M,
                                       int64_t *d_cost, int16_t *d_dec, void *d_work, uint64_t work_bytes,
                                       void *stream, int32_t schedule);

/* Kernel classes of the fill, for rotor_solve_timed. */
#define ROTOR_KERNEL_LEAF 0   /* single-stage cells, Eq. (DP:Init) */
#define ROTOR_KERNEL_DIAG 1   /* pairs inside one 16-stage diagonal block, all splits */
#define ROTOR_KERNEL_MIDDLE 2 /* split points whose operands lie in finished blocks */
#define ROTOR_KERNEL_EDGE 3   /* remaining split points, C_2, gates, final cells */
#define ROTOR_KERNEL_PREP 4   /* gates, prefix sums, value path of every block-diagonal */
#define ROTOR_N_KERNEL_CLASSES 5

typedef struct {
    int32_t launches;          /* kernel launches of this class */
    double ms;                 /* time of this class's launches, from HIP events */
    uint64_t split_candidates; /* C_1 candidates evaluated (split point x budget x pair) */
    uint64_t all_candidates;   /* C_2 candidates evaluated (budget x pair) */
    uint64_t cells;            /* final (cost, decision) cells written */
} rotor_kernel_stats;

/* rotor_solve, plus a breakdown of the fill by kernel class: a HIP event pair
 * is recorded around each run of consecutive launches of one class on one
 * stream (`stream`, or the side stream of the blocked fill), the runs' times
 * summed per class, and the call waits for both streams.  Runs on the two
 * streams overlap, so the class times can add up to more than the fill.
 * stats: HOST array of ROTOR_N_KERNEL_CLASSES entries, overwritten.
 * Summed over the classes, split_candidates is (L^3 - L)/6 (M+1) n_chains and
 * all_candidates L(L-1)/2 (M+1) n_chains.  Same return codes as rotor_solve. */
ROTOR_API int32_t rotor_solve_timed(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost,
                                    int16_t *d_dec, void *d_work, uint64_t work_bytes, void *stream,
                                    rotor_kernel_stats *stats);

/* Algorithm 2 (OptRec): the optimal persistent sequence of the whole chain
 * [1, L] of chain `chain` for each of n_budgets budgets, walked on the device
 * from the decision table that rotor_solve wrote.  The F_none steps of a C_1
 * split stop at stage s'-1 (the stage whose output is stored next; the C_ck
 * cost charges u_f^s .. u_f^{s'-1}).
 *
 *   d_params   DEVICE: the parameters given to rotor_solve.
 *   d_dec      DEVICE: the decision table rotor_solve wrote (same n_chains,
 *              L, M).
 *   d_budgets  DEVICE, n_budgets int64 budgets m (0 <= m <= M).
 *   d_ops      DEVICE, written: n_budgets x cap rotor_op; the sequence of
 *              budget b starts at d_ops + b * cap.  A sequence has at most
 *              L(L+1)/2 + L operations.
 *   d_count    DEVICE, written: n_budgets int64, the sequence length (on
 *              ROTOR_ECAPACITY: the length needed; only cap ops are written).
 *   d_status   DEVICE, written: n_budgets int32, ROTOR_OK, ROTOR_INFEASIBLE
 *              (C(1, L, m) is infinite; count 0), ROTOR_ECAPACITY,
 *              ROTOR_EINVAL (budget out of range), ROTOR_EDOMAIN (the
 *              chain's parameters are outside the domain; count 0) or
 *              ROTOR_ECORRUPT.
 * Asynchronous.  Returns ROTOR_OK once enqueued, ROTOR_EINVAL for bad
 * arguments (including L > ROTOR_MAX_L_RECONSTRUCT), ROTOR_EDEVICE if the
 * launch fails.  Allocates nothing. */
ROTOR_API int32_t rotor_reconstruct(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M,
                                    const int16_t *d_dec, int32_t chain, int32_t n_budgets,
                                    const int64_t *d_budgets, int64_t cap, rotor_op *d_ops, int64_t *d_count,
                                    int32_t *d_status, void *stream);

/* ---- front end: from measured sizes to budgets (host only) --------------- */

/* Discretisation of Section 5.2: for a memory limit of mem_bytes and S slots,
 * every memory size becomes a whole number of slots of mem_bytes / S bytes,
 * rounded up: ceil(v * S / mem_bytes).  The DP then runs with the budget
 * M = S, whatever the limit, and each size is overestimated by less than one
 * slot.
 *
 *   h_params     HOST, read only: [n_chains][6][L] int64 in the layout above,
 *                except that the rows ROTOR_ROW_WA, _WABAR, _OF and _OB hold
 *                sizes in bytes (or any unit of mem_bytes).
 *   h_mem_bytes  HOST, read only: [n_chains] the memory limit of each chain,
 *                > 0; a batch may give the same chain several limits.
 *   slots        S, 1 <= S < 2^28.
 *   h_out        HOST, written: [n_chains][6][L], the time rows copied, the
 *                four size rows in slots.  May be h_params itself.
 * Returns ROTOR_OK; ROTOR_EINVAL for a null pointer, sizes out of range, a
 * limit <= 0 or S out of range; ROTOR_EDOMAIN if an input is negative or a
 * size comes to 2^30 slots or more.  Nothing is written unless ROTOR_OK. */
ROTOR_API int32_t rotor_discretize(const int64_t *h_params, int32_t n_chains, int32_t L, const int64_t *h_mem_bytes,
                                   int64_t slots, int64_t *h_out);

/* Peak memory of the schedule that recomputes nothing -- F_all^1 ..
 * F_all^L, then B^L .. B^1 -- under the memory accounting of Theorem 1
 * (Section 4.2): the chain input is not counted, delta^l has the size of a^l,
 * and during F_all^j the gradient delta^L, abar^1 .. abar^j and o_f^j are
 * live, during B^j delta^j, abar^1 .. abar^j and o_b^j.  This is the memory
 * of the store-everything strategy the experiments of Section 5.3 compare
 * against; every budget at or above it gives the time sum(u_f + u_b).
 *
 *   h_params  HOST, read only: [6][L] int64, one chain (any size unit).
 *   peak      HOST, written.
 * Returns ROTOR_OK, ROTOR_EINVAL (null pointer, L out of range) or
 * ROTOR_EDOMAIN (a negative value). */
ROTOR_API int32_t rotor_store_all_peak(const int64_t *h_params, int32_t L, int64_t *peak);

/* The n budgets equally spaced between 0 (excluded) and top (included), as
 * the experiments of Section 5.3 take 10 limits up to the store-everything
 * memory: budgets[i-1] = floor(i * top / n), i = 1..n.  One rotor_reconstruct
 * call then walks all of them in the same table.
 *   top >= 0, 1 <= n <= 2^20, budgets HOST [n] written.
 * Returns ROTOR_OK or ROTOR_EINVAL. */
ROTOR_API int32_t rotor_even_budgets(int64_t top, int32_t n, int64_t *budgets);

/* Time and peak memory of an operation sequence on the whole chain [1, L],
 * replayed with the operation semantics of Table 1 (Section 3.1) and the
 * memory accounting of Theorem 1 (Section 4.2): at the start the chain input
 * a^0 (not counted) and the gradient delta^L are stored; a forward operation
 * of stage l needs a^{l-1} (F_ck and F_all also accept abar^{l-1}), and F_none
 * replaces a^{l-1} by its output; the peak of a forward is what is stored
 * plus its output (abar^l for F_all, a^l otherwise) plus o_f^l; B^l needs
 * delta^l, abar^l and a^{l-1} or abar^{l-1}, peaks at what is stored plus
 * o_b^l, frees delta^l and abar^l (and a plain a^{l-1}) and stores
 * delta^{l-1}; a^l and delta^l have size w_a^l, abar^l size w_abar^l, and the
 * sequence must end with exactly delta^0 stored.  This is the prediction the
 * DP makes for a sequence, e.g. one rotor_reconstruct returned, in the units
 * of the parameters.
 *
 *   h_params  HOST, read only: [6][L] int64, one chain.
 *   h_ops     HOST, read only: [n_ops] operations.
 *   time, peak  HOST, written: sum of the operations' times, peak memory.
 * Returns ROTOR_OK; ROTOR_EINVAL (null pointer, L out of range, n_ops < 0,
 * an unknown kind or a stage outside 1..L); ROTOR_EDOMAIN (a negative
 * parameter); ROTOR_ESEQUENCE if an operation's input is missing, a value is
 * stored twice or anything but delta^0 is left at the end. */
ROTOR_API int32_t rotor_sequence_cost(const int64_t *h_params, int32_t L, const rotor_op *h_ops, int64_t n_ops,
                                      int64_t *time, int64_t *peak);

#ifdef __cplusplus
}
#endif

#endif /* ROTOR_H */
