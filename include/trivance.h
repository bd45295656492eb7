/*
 * trivance.h -- C ABI of the MI355X (gfx950) emulated Trivance AllReduce.
 *
 * Trivance (Juerss, Addanki, Schmid, arXiv 2602.17254) is an AllReduce for bidirectional rings
 * and tori: at step k every rank exchanges data with the two peers at distance 3^k in opposite
 * directions and reduces both incoming messages together with its own partial result (a "joint
 * reduction"), finishing in log3(n) steps (Sec. 4). This library executes that schedule for n
 * *virtual* ranks whose vectors all live in one GPU's memory: a "send" is a read of another
 * rank's row, and every step is materialised in HBM before the next one starts (the per-step
 * barrier of Sec. 4.3 is a kernel boundary).
 *
 * Conventions for every function:
 *   - return value 0 (TRIVANCE_OK) on success, a negative trivance_status on failure;
 *   - pointers documented as "device" must point to GPU memory of the current HIP device,
 *     pointers documented as "host" to ordinary CPU memory;
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream);
 *   - nothing is retained after return except what a plan owns.
 * Nothing here depends on PyTorch; the Python binding only marshals arguments.
 */
#ifndef TRIVANCE_H
#define TRIVANCE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TRIVANCE_MAX_DIMS 8

/* Opaque, immutable schedule. May be shared by threads and streams once created. */
typedef struct trivance_plan trivance_plan_t;

typedef enum {
    TRIVANCE_LATENCY_OPT = 0,   /* Sec. 4.2: whole segments every step, log3(n) passes        */
    TRIVANCE_BANDWIDTH_OPT = 1, /* Sec. 4.1: reduce-scatter then all-gather, 2 log3(n) passes */
    TRIVANCE_BRUCK_REF = 2      /* Sec. 2.4 / Fig. 1 comparison pattern on a ring: offsets
                                   +3^k and +2*3^k. Congestion counting only; not executable. */
} trivance_variant;

typedef enum { TRIVANCE_F32 = 0, TRIVANCE_I32 = 1 } trivance_dtype;

typedef enum {
    TRIVANCE_ROUTE_SCHEDULED = 0, /* a message travels in the direction of its offset's sign   */
    TRIVANCE_ROUTE_SHORTEST = 1   /* the shorter way round its ring; a tie keeps the sign
                                     (Appendix C's rerouted Bruck; Appendix E)                 */
} trivance_routing;

typedef enum {
    TRIVANCE_PHASE_LATENCY = 0,        /* one step of the latency-optimal variant   */
    TRIVANCE_PHASE_REDUCE_SCATTER = 1, /* one reduce-scatter step (joint reduction) */
    TRIVANCE_PHASE_ALLGATHER = 2       /* one all-gather step (copies only)         */
} trivance_phase;

typedef struct {
    int ndims;                   /* must equal the plan's number of dimensions */
    int dims[TRIVANCE_MAX_DIMS]; /* must equal the plan's sides                 */
    int routing;                 /* a trivance_routing                          */
} trivance_topology;

typedef enum {
    TRIVANCE_OK = 0,
    TRIVANCE_EINVAL = -1,      /* bad argument: NULL pointer, sizes that do not match, ranges  */
    TRIVANCE_EUNSUPPORTED = -2,/* valid request outside what is implemented (see each call)    */
    TRIVANCE_EHIP = -3,        /* the HIP runtime reported an error (launch, copy, allocation) */
    TRIVANCE_ENOMEM = -4,      /* host memory allocation failed                                */
    TRIVANCE_ESIZE = -5,       /* caller-provided output is too small                          */
    TRIVANCE_ESCRATCH = -6     /* request larger than the library's fixed device scratch       */
} trivance_status;

/*
 * trivance_plan -- build the step / peer / block schedule (host only, no GPU work).
 *
 *   n           number of virtual ranks; must equal the product of the sides.
 *   torus_dims  host array of ndims sides, dimension 0 varying fastest in the rank numbering
 *               (rank = x_0 + n_0 * (x_1 + n_1 * (...))). ndims == 0 or torus_dims == NULL
 *               means a ring of n.
 *   variant     a trivance_variant.
 *   out         receives the new plan; release it with trivance_plan_destroy.
 *
 * Schedule (Sec. 4.1 peers pi(r,k) = r -/+ 3^k; Theorem 1 step count; Sec. 5 tori): S = log3(n)
 * steps. On a D-dimensional torus D collectives run concurrently, collective c on segment c of
 * every vector; at global step t collective c works on dimension (c + t) mod D at distance
 * 3^(t div D) (Sec. 5 dimension switching, Appendix B step index t = d + D k). Sides may differ
 * (rectangular tori, which Sec. 5 does not cover); then collective c at step t takes the first
 * dimension, in cyclic order from (c + t) mod D, in which it still has steps left, at distance
 * 3^(steps it already took there). With equal sides both rules coincide.
 *
 * Sides that are not powers of three (Sec. 4.4): a side of s with 3^f < s < 3^(f+1) takes f steps
 * at distances 3^0 .. 3^(f-1) and a final step at d = ceil((s - 3^f) / 2), so ceil(log3 s) steps;
 * S is the sum over the sides, and the dimension of every step follows the rule for unequal sides
 * above. The paper gives no construction of the block sets or partial sums:
 *   - bandwidth-optimal: every block is reduced along one tree per dimension, built so that each
 *     rank forwards each block once per phase (the tree of a side that is a power of three is the
 *     ordinary one). Limits: at most 4 dimensions, sides up to 2200, at most 20 steps, and at
 *     most 768 offset-table entries per step (the lists travel in kernel arguments).
 *   - latency-optimal: a rank keeps its Lemma 2 window and, besides it, the partial sums over
 *     parts of its window that a peer will need from it: in the final step along a side the
 *     peer at +d sends the sum of the top d sources of its window and the peer at -d the sum of
 *     the s - 3^f - d sources beyond the receiver's window on that side (offsets taken in
 *     (-s/2, s/2], so an odd remainder puts the extra source on the + side); each such partial
 *     is formed in earlier steps from the parts of it that lie in the three previous windows.
 *     A rank holds at most 64 partials per collective between passes (more: EUNSUPPORTED); they
 *     live in a caller-provided workspace (trivance_workspace_bytes,
 *     trivance_allreduce_emulated_ws). Limits: at most 4 dimensions, sides up to 2200.
 *
 * Errors: EINVAL for out == NULL, n < 1, ndims < 0, a side < 1, product != n;
 *         EUNSUPPORTED for a side that is not a power of three with the Bruck variant, beyond
 *         the limits above, ndims > TRIVANCE_MAX_DIMS, or TRIVANCE_BRUCK_REF on more than one
 *         dimension.
 */
int trivance_plan(int n, const int* torus_dims, int ndims, int variant, trivance_plan_t** out);

/* Plan option (trivance_plan_ex): message-contiguous block placement. */
#define TRIVANCE_PLACE_BY_SCHEDULE 1u

/*
 * trivance_plan_ex -- trivance_plan with options.
 *   flags  0, or TRIVANCE_PLACE_BY_SCHEDULE: block j of every segment lies at the granule range of
 *          position pos_c(j) instead of the j-th one (see trivance_block_range). pos_c(j) spells
 *          the base-3 digits of block j's coordinates in the order collective c's steps fix them
 *          (each step fixes the next digit of the coordinate of the dimension it works on; with
 *          equal sides step t fixes digit t div D of dimension (c + t) mod D), most significant
 *          first. The blocks a rank keeps after each reduce-scatter step (Sec. 4.3 closed form)
 *          and every message are then one contiguous range of positions. Power-of-three sides,
 *          bandwidth-optimal variant only (EUNSUPPORTED otherwise). The option changes
 *          which elements share a block, hence an element's fp32 summation tree; int32 results
 *          are the same exact sums.
 * Errors: those of trivance_plan, and EINVAL for unknown flag bits.
 */
int trivance_plan_ex(int n, const int* torus_dims, int ndims, int variant, unsigned flags,
                     trivance_plan_t** out);

/* Release a plan (NULL is ignored). */
void trivance_plan_destroy(trivance_plan_t* plan);

/* Number of steps S = log3(n) (>= 0), or a negative status for plan == NULL. */
int trivance_plan_num_steps(const trivance_plan_t* plan);

/* Number of passes (kernel-materialised steps): S for latency-optimal and Bruck, 2 S for
 * bandwidth-optimal (S reduce-scatter steps, then S all-gather steps in reverse order). */
int trivance_plan_num_passes(const trivance_plan_t* plan);

/*
 * trivance_plan_step -- introspection of one pass for one collective.
 *   phase    <- a trivance_phase
 *   dim      <- torus dimension used by this collective in this pass
 *   distance <- peer distance of this collective in this pass (3^(t div D) for equal sides; the
 *               tree step's distance for a side that is not a power of three)
 * Any output pointer may be NULL. EINVAL if pass or collective is out of range.
 */
int trivance_plan_step(const trivance_plan_t* plan, int pass, int collective, int* phase,
                       int* dim, int* distance);

/* Global step index t (Sec. 5, Appendix B: t = d + D k) that pass `pass` materialises: 0 .. S-1
 * for the latency-optimal and reduce-scatter passes, S-1 .. 0 for the all-gather passes (Sec. 4.1
 * reverse order). Returns t >= 0, or EINVAL for a NULL plan or a pass out of range. */
int trivance_plan_step_index(const trivance_plan_t* plan, int pass);

/*
 * trivance_block_range -- element range [begin, end) of block `block` in segment `collective`
 * for vectors of `elems` elements. The paper assumes blocks of m/n (Sec. 2.2, 4.1); the rounding
 * rule used here: 64-element granules, G = ceil(elems / 64); segment c holds granules
 * [floor(c G / D), floor((c+1) G / D)); block j of a G_c-granule segment holds its granules
 * [floor(j G_c / n), floor((j+1) G_c / n)); bounds are clipped at elems. Blocks may be empty.
 * Plans made with TRIVANCE_PLACE_BY_SCHEDULE place block j at the range of position pos_c(j)
 * (trivance_plan_ex) instead of the j-th range.
 * block == -1 returns the whole segment. Block j is owned (finished) by rank j.
 * EINVAL for a NULL output, elems < 0, or an index out of range.
 */
int trivance_block_range(const trivance_plan_t* plan, int64_t elems, int collective, int block,
                         int64_t* begin, int64_t* end);

/*
 * trivance_algorithmic_bytes -- bytes the step-by-step schedule must move through memory for one
 * AllReduce of `elems` elements per rank (each participating location read once and each output
 * written once per pass). Latency-optimal: 2 S n elems w (with partial sums on sides that are not
 * powers of three: every partial a rank holds before a pass read once, every one after it
 * written once). Bandwidth-optimal: reduce-scatter step t
 * reads n elems w / 3^t and writes a third of that; all-gather step t reads n elems w / 3^(t+1)
 * and writes twice that; in total 3.5 w elems (n - 1) for divisible sizes (the exact sum over the
 * actual blocks is returned). Sides that are not powers of three: in every tree step each
 * receiving rank reads its own partial and each sending child and writes once (reduce-scatter),
 * or reads once and writes each child (all-gather). w = 4 for both dtypes. Negative status on bad
 * arguments.
 */
int64_t trivance_algorithmic_bytes(const trivance_plan_t* plan, int64_t elems, int dtype);

/* Same accounting for a single pass (0 <= pass < num_passes). */
int64_t trivance_pass_bytes(const trivance_plan_t* plan, int64_t elems, int dtype, int pass);

/*
 * trivance_allreduce_emulated -- run the whole schedule, in place, on n virtual ranks.
 *
 *   buffers  device array of n * elems values, rank-major: rank r's vector is
 *            buffers[r * elems .. (r + 1) * elems). Caller-owned; updated in place.
 *   n        number of ranks (must match the plan).
 *   elems    elements per rank (>= 0).
 *   dtype    TRIVANCE_F32 or TRIVANCE_I32 (int32 adds wrap modulo 2^32).
 *   plan     a latency- or bandwidth-optimal plan.
 *   stream   hipStream_t (NULL = default stream).
 *
 * Semantics (Sec. 2.2, 4.1-4.3, 5): integer results equal the exact column sums on every rank.
 * Float results follow the schedule: each joint reduction computes (own + left) + right with
 * left the peer at -distance, in IEEE fp32 round-to-nearest-even, no fused or reordered adds
 * (for sides that are not powers of three a term is skipped when no child sends from that side).
 * The latency-optimal variant leaves ranks with (legitimately) different float bits; the
 * bandwidth-optimal one leaves identical bits on every rank.
 *
 * Asynchronous: all passes are enqueued on `stream` and the call returns; execution errors
 * surface on stream synchronisation. No device memory is allocated, no memory is set and no host
 * synchronisation happens, so the call can be captured into a HIP graph (replays reproduce it).
 * n == 1 or elems == 0 is a valid no-op. Calls that overlap on the same buffers race; calls on
 * different buffers may run concurrently on different streams.
 * Plans whose trivance_workspace_bytes is not zero (latency-optimal with a side that is not a
 * power of three) need trivance_allreduce_emulated_ws; this form returns ESIZE for them.
 * Errors: EINVAL (NULL plan/buffers with elems > 0, n mismatch, elems < 0, bad dtype),
 * EUNSUPPORTED (a Bruck plan, sizes beyond 32-bit work-unit counts), ESIZE (a plan that needs a
 * workspace), EHIP (launch failure).
 */
int trivance_allreduce_emulated(void* buffers, int n, int64_t elems, int dtype,
                                const trivance_plan_t* plan, void* stream);

/* Same, running only passes [pass_begin, pass_end) (0 <= begin <= end <= num_passes); used to
 * inspect or resume the state between steps. Running all ranges back to back equals one full
 * call. */
int trivance_allreduce_emulated_steps(void* buffers, int n, int64_t elems, int dtype,
                                      const trivance_plan_t* plan, void* stream, int pass_begin,
                                      int pass_end);

/*
 * trivance_workspace_bytes -- device workspace an AllReduce of `elems` elements per rank needs
 * with this plan: 0 for every plan that runs in place (all bandwidth-optimal plans and the
 * latency-optimal ones whose sides are powers of three). A latency-optimal plan with a side that
 * is not a power of three keeps up to P partial sums per rank between passes (P = the plan's
 * largest slot count) in two halves of P * n * elems values each (one when the plan has at most
 * two steps): 4 bytes per value for both dtypes. Negative status on bad arguments.
 */
int64_t trivance_workspace_bytes(const trivance_plan_t* plan, int64_t elems, int dtype);

/*
 * trivance_allreduce_emulated_ws -- trivance_allreduce_emulated with a caller-owned device
 * workspace of at least trivance_workspace_bytes(plan, elems, dtype) bytes (NULL with 0 bytes is
 * fine for plans that need none). The workspace holds the partial sums between passes (Sec. 4.4,
 * latency-optimal: see trivance_plan); its contents on entry do not matter and are left
 * undefined. A 16-byte aligned workspace keeps the 16-byte vector path. Calls that share a
 * workspace or buffers race. Like the plain form it enqueues kernel launches only (a one-pass
 * program copies its result back with a kernel), so it can be captured into a HIP graph.
 * Errors: those of trivance_allreduce_emulated, and ESIZE for a workspace below the required
 * size.
 */
int trivance_allreduce_emulated_ws(void* buffers, int n, int64_t elems, int dtype,
                                   const trivance_plan_t* plan, void* workspace,
                                   int64_t workspace_bytes, void* stream);

/* Same, running only passes [pass_begin, pass_end). Consecutive ranges must use the same
 * workspace: it carries the partial sums from one range to the next. */
int trivance_allreduce_emulated_steps_ws(void* buffers, int n, int64_t elems, int dtype,
                                         const trivance_plan_t* plan, void* workspace,
                                         int64_t workspace_bytes, void* stream, int pass_begin,
                                         int pass_end);

/*
 * trivance_congestion -- per-pass, per-directed-link message counts (Sec. 2.1: c_k = number of
 * chunks sharing a link), computed on the GPU and copied to a host array. Synchronous.
 *
 *   topo       sides (must equal the plan's) and routing; NULL = the plan's sides, scheduled
 *              routing.
 *   loads      host int64 array [passes][n][2 D]; entry [p][r][2d] counts messages crossing the
 *              link that leaves rank r towards +d in pass p, [p][r][2d+1] towards -d.
 *   loads_len  number of entries available.
 *
 * Every rank sends one message per collective to each peer of the active dimension; for a side
 * that is not a power of three, only towards the sides from which some child of that
 * dimension's tree sends in the step (all-gather steps retrace the messages, so the directions
 * swap).
 *
 * loads == NULL returns the required length (positive). ESIZE if loads_len is too small,
 * EUNSUPPORTED for a side above 6561 or 2^31 and more (pass, dimension, line) triples. Allocates
 * and frees a temporary device buffer.
 */
int64_t trivance_congestion(const trivance_plan_t* plan, const trivance_topology* topo,
                            int64_t* loads, int64_t loads_len);

/* Asynchronous form writing the same array into caller-owned device memory `loads_dev` on
 * `stream`; allocates nothing. */
int trivance_congestion_device(const trivance_plan_t* plan, const trivance_topology* topo,
                               int64_t* loads_dev, int64_t loads_len, void* stream);

/*
 * trivance_congestion_noalloc -- trivance_congestion for callers that cannot allocate device
 * memory (serving loops and harnesses that forbid hipMalloc): the same host array, the same
 * arguments, NULL loads returning the required length and ESIZE as there, but computed into a
 * fixed device scratch that the library holds, one per GPU, from the first call on that GPU
 * until the process ends. Calls no hipMalloc, hipFree or other allocating routine.
 * Limit: at most 2^20 entries (passes x n x 2 D; 8 MiB of scratch); larger plans return
 * TRIVANCE_ESCRATCH before any GPU work. Synchronous. Every call on one GPU uses that GPU's
 * scratch, so calls that overlap on one GPU (from several host threads) race; calls on
 * different GPUs do not. Errors: those of trivance_congestion, and ESCRATCH.
 */
int64_t trivance_congestion_noalloc(const trivance_plan_t* plan, const trivance_topology* topo,
                                    int64_t* loads, int64_t loads_len);

/* Result of trivance_cost_model (all times in the units of alpha and beta). */
typedef struct {
    double total;        /* C(m, A) = latency + transmission                                     */
    double latency;      /* passes x alpha                                                       */
    double transmission; /* beta x the sum over passes of the busiest directed link's bytes      */
    double theta;        /* that sum relative to m / D: the transmission-delay factor of Tables 1
                            and 2 (relative to m on a ring)                                     */
    int passes;          /* number of passes, i.e. steps(A)                                      */
} trivance_cost_result;

/*
 * trivance_cost_model -- the congestion-aware cost model of Sec. 2.1 for this plan (host only,
 * synchronous, no GPU work):
 *     C(m, A) = steps(A) alpha + sum over passes of beta m_k c_k,
 * where m_k c_k is read per directed link: the bytes of every message crossing the pass's busiest
 * link. Every rank of a collective sends one message to each side along its active dimension over
 * the pass's distance, so each directed link of that dimension carries `distance` of them per
 * collective. Message sizes for m bytes per rank split into D segments of m / D and n blocks of
 * m / (n D): the whole segment (latency-optimal, Sec. 4.2); n / 3^(t+1) blocks at step t of both
 * phases (bandwidth-optimal, Sec. 4.1, Lemma 1); on sides that are not powers of three the blocks
 * the tree forwards that way in the step (Sec. 4.4). Blocks are taken as exact fractions of m
 * (the partition's 64-element rounding is not modelled). Trivance's distances are below half
 * their side, so the scheduled direction is the shortest path (Appendix E).
 *
 *   bytes_per_rank   m, the AllReduce size per rank, in bytes (>= 0)
 *   alpha            per-step start-up latency (e.g. seconds), >= 0
 *   beta             transmission time per byte of one link (e.g. seconds per byte), >= 0
 *   pass_link_bytes  optional host array [pass_len]: receives the busiest link's bytes per pass
 *   out              receives the totals
 * Errors: EINVAL for a NULL plan or out or a negative (or NaN) m, alpha or beta; ESIZE if
 * pass_link_bytes is given and pass_len < the number of passes; EUNSUPPORTED for a Bruck plan.
 */
int trivance_cost_model(const trivance_plan_t* plan, double bytes_per_rank, double alpha,
                        double beta, double* pass_link_bytes, int pass_len,
                        trivance_cost_result* out);

/*
 * trivance_fill_hash_uniform -- input generator (not part of the AllReduce): writes U(-1, 1)
 * fp32 values to the device array `buffers` of n * elems floats, value (r, e) being the k-th
 * output of SplitMix64 (Steele, Lea, Flood 2014) started from state 0 with
 * k = seed * 2^40 + r * elems + e + 1, mapped to (h >> 40) * 2^-23 - 1. Asynchronous on stream.
 */
int trivance_fill_hash_uniform(void* buffers, int n, int64_t elems, uint64_t seed, void* stream);

/*
 * trivance_copy_device -- benchmark helper (not part of the AllReduce): copies `bytes` bytes from
 * device memory `src` to device memory `dst` with a plain streaming kernel (per lane one 16-byte
 * non-temporal load and one streaming store with the cache policy of the step kernels' large
 * passes, one-wave workgroups), the simplest kernel with the step kernels' access granularity.
 * Its rate is the practical HBM ceiling reported beside them.
 * Asynchronous on stream. EINVAL unless bytes >= 0, bytes % 16 == 0, both pointers are 16-byte
 * aligned and the two ranges do not overlap; bytes == 0 does nothing.
 */
int trivance_copy_device(void* dst, const void* src, int64_t bytes, void* stream);

/*
 * trivance_plan_with_dispatch_limit -- a new, independent plan equal to `plan` except that every
 * launch made with it is issued as dispatches of at most `work_items` work-items (the default and
 * maximum is 2^31). A dispatch carries its grid size as a 32-bit count of work-items, so every
 * launch of this library whose grid is larger is issued as consecutive dispatches of whole
 * workgroups on the same stream; the results do not depend on the split. A smaller limit only
 * adds dispatches: it exists to exercise the split at small sizes. `plan` is not modified and
 * stays valid; release `*out` with trivance_plan_destroy.
 * Errors: EINVAL for a NULL plan or out, or work_items outside [1024, 2^31]; ENOMEM.
 */
int trivance_plan_with_dispatch_limit(const trivance_plan_t* plan, int64_t work_items,
                                      trivance_plan_t** out);

/* Static description of a status code. */
const char* trivance_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* TRIVANCE_H */
