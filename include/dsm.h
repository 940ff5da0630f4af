/*
 * dsm.h - distributed sign momentum with local steps on one MI355X (gfx950).
 *
 * The method (arXiv 2411.17866, Section 2, Algorithm 1) minimises
 * f(x) = (1/n) sum_i f_i(x), x in R^d (Eq. (1)), with n workers.  Each outer
 * iteration t, every worker i takes tau = H local steps of a base optimizer
 * (Eq. (4)); then the replicas are averaged (the all-reduce step), a global
 * sign-momentum step updates the model and the global momentum (Eqs. (6)-(8))
 * and the new model is copied back to every replica (synchronisation step).
 *
 * On one GPU the n workers are n replicas resident in HBM, and the all-reduce
 * is a per-element sum over the replicas in worker order.  x in R^d is a list
 * of tensors; they live concatenated in one flat fp32 arena per buffer, each
 * tensor starting at a multiple of 64 elements (256 bytes; 1024 elements with
 * blocked replicas).  dsm_layout gives the arena length (d_pad) and every
 * tensor's offset.
 *
 * Conventions for every entry point:
 *  - All arithmetic state is fp32.  Hyperparameters are fp32 numbers.
 *  - Device pointers are allocated and owned by the caller (for instance as
 *    torch tensors), must be 256-byte aligned, and must stay allocated and
 *    unmoved for the lifetime of the context.  The library never allocates
 *    or frees device memory.
 *  - Calls that touch the GPU only enqueue work on the caller's stream and
 *    return; completion is observed with the caller's stream or event
 *    synchronisation.  dsm_read_bounds and dsm_destroy synchronise the stream.
 *  - A status is returned; no exception crosses the boundary.  Argument and
 *    state errors are detected on the host before anything is enqueued, and
 *    then nothing is modified.  dsm_last_error gives the message.
 *  - A context is not thread-safe; use one context per thread or lock.
 *    Contexts may share the model buffers (they then take turns on the same
 *    state) but never a workspace.
 */
#ifndef DSM_H
#define DSM_H

#include <stdint.h>

#if defined(__GNUC__)
#define DSM_API __attribute__((visibility("default")))
#else
#define DSM_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dsm_ctx dsm_ctx; /* opaque, host-side */

typedef enum dsm_status {
    DSM_OK = 0,
    DSM_ERR_INVALID_ARG = 1, /* bad pointer, size, alignment or hyperparameter */
    DSM_ERR_STATE = 2,       /* call out of the order Algorithm 1 requires */
    DSM_ERR_HIP = 3,         /* HIP runtime error (no device, launch, copy) */
    DSM_ERR_UNSUPPORTED = 4  /* valid request the library does not implement */
} dsm_status;

/* Base optimizer of the local steps (Section 2, "any base optimizer"). */
typedef enum dsm_base {
    DSM_BASE_ADAMW = 0,        /* Algorithm 2 (Appendix A) */
    DSM_BASE_SGD_MOMENTUM = 1  /* Algorithm 3 (Appendix A), Polyak momentum */
} dsm_base;

/* The sign applied in the global step (Eq. (7)). */
typedef enum dsm_sign {
    DSM_SIGN_DET = 0,       /* sign(u), with sign(0) = 0 */
    DSM_SIGN_RAND_FLIP = 1, /* randomized sign of Eq. (9) (Section 3.1) */
    DSM_SIGN_RAND_ZERO = 2  /* randomized sign of Eq. (10) (Section 3.1) */
} dsm_sign;

/* The global update (dsm_global_hparams.rule): the method's sign momentum,
 * or one of the ablation variants of its global step. */
typedef enum dsm_global_rule {
    DSM_RULE_SIGN_MOMENTUM = 0, /* Eqs. (6)-(8) */
    DSM_RULE_LOOKAHEAD = 1,     /* Section 4.1: Eq. (7) with u in place of sign(u):
                                   x <- x - eta gamma (u + lambda x); lambda = 0 is the
                                   paper's Lookahead */
    DSM_RULE_SIGNED_SLOWMO = 2, /* Section 4.1: u = b1 m + ((1-b1)/gamma) sign(delta),
                                   x <- x - eta gamma (u + lambda x), Eq. (8) unchanged */
    DSM_RULE_GLOBAL_ADAMW = 3   /* Algorithm 7 (Appendix C): AdamW with learning rate
                                   eta on g = delta/gamma, bias corrections 1 - b^(t+1);
                                   needs buffers.v */
} dsm_global_rule;

/* How the n worker replicas x_rep share their buffer (dsm_problem.replica_layout).
 * The other per-worker buffers (g_rep, s1_rep, s2_rep) hold n contiguous
 * copies, except in DSM_REPLICAS_STATE_BLOCKED. */
typedef enum dsm_replica_layout {
    DSM_REPLICAS_CONTIGUOUS = 0, /* copy i at element offset i * d_pad */
    DSM_REPLICAS_BLOCKED = 1,    /* 64 KiB blocks interleaved by worker: element e of
                                    copy i at ((e / 16384) * n + i) * 16384 + e % 16384.
                                    A work-group's n replica accesses then fall in one
                                    n * 64 KiB span instead of n spans d_pad apart; the
                                    global step and the synchronisation, which write
                                    every replica, keep their bandwidth in every
                                    physical placement.  d_pad is a multiple of 16384
                                    and tensors start on multiples of 1024 elements. */
    DSM_REPLICAS_STATE_BLOCKED = 2 /* the replicas and their state in one allocation of
                                    B * n * d_pad floats (B = 4 for AdamW, 3 for SGD) in
                                    16 KiB blocks: block b holds the n x_rep copies, then
                                    the n g_rep, the n s1_rep and (AdamW) the n s2_rep
                                    copies of elements [4096 b, 4096 b + 4096), so element
                                    e of copy i of buffer j is at ((e / 4096) * B * n +
                                    j * n + i) * 4096 + e % 4096.  Pass x_rep = the
                                    allocation, g_rep = x_rep + n * 4096, s1_rep = x_rep
                                    + 2 n * 4096, s2_rep = x_rep + 3 n * 4096.  The
                                    streams a work-group touches then share one
                                    B * n * 16 KiB span, and the local steps take the
                                    same piece of every worker in turn, so they sweep
                                    whole blocks; local steps measured faster at n = 4
                                    and n = 8.  d_pad is a multiple of 4096, tensors
                                    start on multiples of 1024 elements. */
} dsm_replica_layout;
#define DSM_REPLICA_BLOCK_ELEMS 16384
#define DSM_STATE_BLOCK_ELEMS 4096

/* The problem of Eq. (1): x in R^d given as n_tensors tensors. */
typedef struct dsm_problem {
    int32_t n_workers;     /* n, 1..64 */
    int32_t local_steps;   /* tau = H >= 1, local steps per outer iteration */
    int32_t n_tensors;     /* >= 0 */
    int32_t base;          /* dsm_base */
    const int64_t* numel;  /* host array [n_tensors], each in [0, 2^34) */
    const uint8_t* decay;  /* host array [n_tensors]: 1 = weight decay applies
                              (local and global); NULL = every tensor decays */
    int32_t replica_layout; /* dsm_replica_layout of x_rep */
} dsm_problem;

/* Device buffers, all fp32 arenas of d_pad elements per copy.  The replica
 * buffers hold n copies (copy i of g_rep, s1_rep, s2_rep at element offset
 * i * d_pad, x_rep as problem->replica_layout says; all four as that layout
 * says in DSM_REPLICAS_STATE_BLOCKED). */
typedef struct dsm_buffers {
    float* x;          /* [d_pad]      global model x_{t,0} (in/out) */
    float* m;          /* [d_pad]      global momentum m_t (zeroed by init) */
    float* x_rep;      /* [n * d_pad]  worker replicas x^(i)_{t,k} */
    float* g_rep;      /* [n * d_pad]  worker direction inputs (gradients),
                          written by the caller before each local step */
    float* s1_rep;     /* [n * d_pad]  AdamW first moment / Polyak momentum */
    float* s2_rep;     /* [n * d_pad]  AdamW second moment; NULL for SGD */
    float* u_scratch;  /* [d_pad]      u_{t+1} staging for the randomized
                          sign; may be NULL if it is never used */
    void* workspace;   /* device, >= workspace_bytes from dsm_layout; holds the
                          context's chunk table and the randomized sign's bound
                          words, so one per context */
    int64_t workspace_bytes;
    void* stream;      /* hipStream_t all work is enqueued on (NULL = default) */
    float* v;          /* [d_pad]      global second moment of DSM_RULE_GLOBAL_ADAMW
                          (zeroed by init); may be NULL if that rule is never used */
} dsm_buffers;

/* Local hyperparameters (Algorithm 2 / Algorithm 3). */
typedef struct dsm_local_hparams {
    float lr;            /* gamma_t of Eq. (4), > 0 */
    float beta1;         /* AdamW beta1, or the Polyak momentum coefficient */
    float beta2;         /* AdamW beta2 (unused for SGD) */
    float eps;           /* AdamW epsilon (unused for SGD) */
    float weight_decay;  /* AdamW decoupled lambda on decayed tensors */
} dsm_local_hparams;

/* Global hyperparameters (Eqs. (6)-(8)). */
typedef struct dsm_global_hparams {
    float gamma;     /* gamma_t, the local learning rate of this round, > 0 */
    float eta;       /* global learning rate eta >= 0 */
    float beta1;     /* beta1 in [0, 1], Eq. (6) */
    float beta2;     /* beta2 in [0, 1], Eq. (8) */
    float lambda;    /* decoupled weight decay lambda >= 0, Eq. (7) */
    int32_t mode;    /* dsm_sign; the variants take DSM_SIGN_DET only */
    uint64_t seed;   /* Philox key of the randomized sign */
    int32_t rule;    /* dsm_global_rule */
    float eps;       /* epsilon of DSM_RULE_GLOBAL_ADAMW (Algorithm 7), >= 0 */
} dsm_global_hparams;

/*
 * dsm_layout - host only; enqueues nothing.
 * Computes the arena layout for a problem: *arena_elems = d_pad, the length
 * of one arena copy; tensor_offsets[p] = element offset of tensor p (the
 * caller provides an array of n_tensors entries, or NULL); and
 * *workspace_bytes = device workspace the context needs: the tensor chunk
 * table, and for the randomized sign the per-tensor bounds with their
 * first-level partial maxima (4 bytes per 1024 elements).  Any output may be
 * NULL.
 * Errors: DSM_ERR_INVALID_ARG for an invalid problem.
 */
DSM_API dsm_status dsm_layout(const dsm_problem* problem, int64_t* arena_elems,
                      int64_t* tensor_offsets, int64_t* workspace_bytes);

/*
 * dsm_init - Algorithm 1 initialisation: m_0 = 0, every replica x^(i)_{0,0} =
 * x_{0,0} (the caller has written x), and the base-optimizer state of every
 * worker is zero (Algorithms 2 and 3 start from m_0 = v_0 = 0).
 * Creates *out (host memory only), uploads the chunk table into the caller's
 * workspace and enqueues the initialisation kernel on buffers->stream.
 * Errors: DSM_ERR_INVALID_ARG (problem, NULL or misaligned pointers, small
 * workspace); DSM_ERR_HIP (no device, copy or launch failure).
 *
 * Resume.  A context keeps no state beyond the caller's buffers and the
 * explicit counters (s, t, seed), so a run saved at a round boundary resumes
 * exactly, in any allocation:
 *   1. write the saved x;
 *   2. call dsm_init;
 *   3. after it on the stream, write back m, s1_rep, s2_rep and v;
 *   4. continue with the saved s and t.
 * A round boundary is the point after dsm_global_step, dsm_round_end or
 * dsm_sync.  The replicas need not be saved: at a round boundary they equal
 * x, or are stale after broadcast = 0, which is the same thing.
 */
DSM_API dsm_status dsm_init(const dsm_problem* problem, const dsm_buffers* buffers,
                    dsm_ctx** out);

/*
 * dsm_init_static - dsm_init for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the context's workspace and the randomized sign's u staging
 * live in a static array of the library, 64 MiB on each GPU it runs on, held
 * until the process ends.  buffers->workspace, workspace_bytes and u_scratch
 * are ignored; every other buffer is the caller's, as for dsm_init.  Nothing
 * is allocated; the call uploads the chunk table and launches the
 * initialisation kernel on buffers->stream like dsm_init.
 * Limit: workspace_bytes (dsm_layout) rounded up to 256, plus 4 * d_pad
 * rounded up to 256, at most 64 MiB (about 16M parameters).
 * One such context may be alive per device at a time, since they would share
 * the array: another dsm_init_static on that device fails until dsm_destroy.
 * Calls on that context from several threads or streams at once race on the
 * array, as they would on a workspace.
 * Errors: as dsm_init; DSM_ERR_INVALID_ARG when the problem exceeds the limit;
 * DSM_ERR_STATE while another context made by dsm_init_static is alive on
 * the current device.
 */
DSM_API dsm_status dsm_init_static(const dsm_problem* problem, const dsm_buffers* buffers,
                                   dsm_ctx** out);

/*
 * dsm_local_step - one local step of Eq. (4), x^(i) <- x^(i) - gamma_t d^(i),
 * with d^(i) from the base optimizer (Algorithm 2 or 3) applied to the
 * direction input g_rep of worker `worker` (0..n-1), or of every worker in
 * one launch when worker == -1.  `step` is the AdamW bias-correction count
 * s >= 1 (ignored for SGD); the caller passes it so that restarts are exact.
 * Per element, in fp32 with one rounding per operation:
 *   AdamW: m = b1*m + (1-b1)*g; v = b2*v + (1-b2)*(g*g);
 *          x = x - lr*((m/(1-b1^s)) / (sqrt(v/(1-b2^s)) + eps) + wd_p*x)
 *   SGD:   m = b1*m + g;  x = x - lr*m
 * with wd_p = weight_decay on decayed tensors, else 0.
 * After a global step with broadcast = 0 a worker's replica is stale: its
 * next local step reads the new global model x in place of the replica (the
 * synchronisation step of Algorithm 1 folded into this step) and writes the
 * replica, which saves the broadcast's n replica writes.
 * Errors: DSM_ERR_INVALID_ARG (worker, step, hyperparameters);
 * DSM_ERR_STATE (the worker already took H local steps this round);
 * DSM_ERR_HIP.
 */
DSM_API dsm_status dsm_local_step(dsm_ctx* ctx, int32_t worker, int64_t step,
                          const dsm_local_hparams* hp);

/*
 * dsm_global_step - Algorithm 1 all-reduce and global step of outer
 * iteration t, fused in one pass (for the randomized sign two, with the
 * per-tensor bound reduced in between):
 *   delta = (1/n) sum_{i=0}^{n-1} (x - x^(i))        (worker order)
 *   u     = b1*m + ((1-b1)/gamma)*delta               Eq. (6)
 *   x     = x - (eta*gamma)*(S(u) + lambda_p*x)       Eq. (7)
 *   m     = b2*m + ((1-b2)/gamma)*delta               Eq. (8), old m
 * S = sign (sign(0) = 0), or the randomized sign of Eq. (9) / Eq. (10) with
 * bound B_p = max_j |u_j| over tensor p and uniforms U = (w >> 8) 2^-24 from
 * Philox4x32-10 keyed by `seed` with counter (j div 4, p, t, 1), word j mod 4
 * (j = index inside the tensor); S keeps sign(u) exactly when U < the
 * equation's probability.  Section 3.1 defines the randomized sign only for a
 * finite bound: a tensor whose B_p is NaN or infinite (it holds a non-finite
 * u) gets S = NaN, so its new x is NaN at every element (dsm_read_bounds
 * shows which tensors).  When broadcast != 0 every replica is set to the
 * new x (synchronisation step); otherwise the replicas are left stale and
 * each worker's next local step reads x (see dsm_local_step), or dsm_sync
 * copies x into them.  The randomized modes need buffers->u_scratch.
 * hp->rule selects an ablation variant of the global update instead
 * (deterministic, same fused pass; Global AdamW also reads and writes
 * buffers->v).
 * Errors: DSM_ERR_INVALID_ARG (t outside [0, 2^32), hyperparameters, mode,
 * unknown rule, a randomized mode with a variant rule, missing u_scratch or
 * v); DSM_ERR_STATE (some worker has not taken exactly H
 * local steps since the last synchronisation); DSM_ERR_HIP.
 */
DSM_API dsm_status dsm_global_step(dsm_ctx* ctx, int64_t t, const dsm_global_hparams* hp,
                           int32_t broadcast);

/*
 * dsm_round_end - the end of outer iteration t of Algorithm 1 in one pass:
 * local step H of every worker (as dsm_local_step(ctx, -1, step, local_hp))
 * fused with the all-reduce and global step (as dsm_global_step(ctx, t,
 * global_hp, broadcast)).  Each worker's step-H replica value is folded into
 * the worker-order sum of Eq. (6)'s difference in registers and is never
 * stored or read back; the base-optimizer state of step H is stored.  The
 * results are bit-identical to the two separate calls.  With broadcast = 0
 * the replicas are left stale (read as x by the next local step), which
 * with the fusion saves 4n + 4n bytes per element per round.
 * Errors: as dsm_local_step and dsm_global_step; DSM_ERR_STATE unless every
 * worker has taken exactly H - 1 local steps this round; DSM_ERR_UNSUPPORTED
 * for a rule other than DSM_RULE_SIGN_MOMENTUM (use the two separate calls).
 */
DSM_API dsm_status dsm_round_end(dsm_ctx* ctx, int64_t step, const dsm_local_hparams* local_hp,
                                 int64_t t, const dsm_global_hparams* global_hp,
                                 int32_t broadcast);

/*
 * dsm_sync - the synchronisation step of Algorithm 1 on its own: every
 * replica is set to x (bit-identical copies), and the local step counts of
 * the round restart at zero.  Errors: DSM_ERR_INVALID_ARG, DSM_ERR_HIP.
 */
DSM_API dsm_status dsm_sync(dsm_ctx* ctx);

/*
 * dsm_read_bounds - copies the per-tensor bounds B_p of the last randomized
 * global step (Eqs. (9)/(10)) into host_B (host memory, caller-owned, room for
 * capacity floats; n_tensors of them are written) and synchronises the stream.
 * A bound that is NaN or infinite marks a tensor whose randomized sign was
 * undefined (a non-finite u in it) and whose step made x NaN.
 * Errors: DSM_ERR_STATE if the last global step was not randomized;
 * DSM_ERR_INVALID_ARG for a NULL context or output, or capacity < n_tensors
 * (nothing is written); DSM_ERR_HIP.
 */
DSM_API dsm_status dsm_read_bounds(dsm_ctx* ctx, float* host_B, int32_t capacity);

/*
 * dsm_test_philox - diagnostic: writes Philox4x32-10 blocks for counters
 * (q0 + b, tensor, t, 1), b = 0..count-1, under key `seed`, as 4*count
 * uint32 words to device memory dev_out (caller-owned, 4-byte aligned), on
 * `stream`.  The same generator the randomized sign uses.
 * Errors: DSM_ERR_INVALID_ARG (NULL output, count < 0, q0 + count > 2^32,
 * t outside [0, 2^32)); DSM_ERR_HIP.
 */
DSM_API dsm_status dsm_test_philox(uint64_t seed, uint32_t tensor, int64_t t, int64_t q0,
                           int64_t count, uint32_t* dev_out, void* stream);

/*
 * dsm_test_stream - diagnostic: streams n_elems fp32 elements of the device
 * buffer dev_buf (caller-owned, 256-byte aligned) with the access shape of the
 * library's kernels: one piece of DSM_PIECE_ELEMS elements per 256-thread
 * work-group, 16-byte nontemporal loads or stores, consecutive lanes on
 * consecutive 16-byte groups.  It measures the device's pure read and pure
 * write rates, and calibrates byte counters against the library's own access
 * shape.  It is a measurement aid, not a step of the method.
 *   DSM_STREAM_READ:  reads every element; for each piece k whose elements'
 *                     32-bit patterns XOR to `pattern`, writes 1 to
 *                     dev_words[k] (caller-owned, n_elems / DSM_PIECE_ELEMS
 *                     words); no other word is written.  With a pattern that
 *                     no piece matches, the kernel only reads;
 *   DSM_STREAM_WRITE: writes the float whose bit pattern is `pattern` to
 *                     every element (dev_words unused).
 * Enqueued on `stream`.  Errors: DSM_ERR_INVALID_ARG (unknown kind, n_elems
 * not a non-negative multiple of DSM_PIECE_ELEMS or beyond one grid
 * dimension, NULL or misaligned buffers); DSM_ERR_UNSUPPORTED (a build whose
 * work-group shape knobs give another piece size); DSM_ERR_HIP.
 */
#define DSM_PIECE_ELEMS 1024
typedef enum dsm_stream_kind { DSM_STREAM_READ = 0, DSM_STREAM_WRITE = 1 } dsm_stream_kind;
DSM_API dsm_status dsm_test_stream(int32_t kind, float* dev_buf, int64_t n_elems,
                                   uint32_t* dev_words, uint32_t pattern, void* stream);

/*
 * dsm_destroy - synchronises the context's stream and frees the context's
 * host memory.  The caller's device buffers are untouched.  NULL is a no-op.
 */
DSM_API dsm_status dsm_destroy(dsm_ctx* ctx);

/*
 * dsm_last_error - message of the last failed call on ctx, or, for ctx ==
 * NULL, of the last failed call on this thread.  Empty string if none.  The
 * pointer stays valid until the next call on the same context or thread.
 */
DSM_API const char* dsm_last_error(const dsm_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* DSM_H */
