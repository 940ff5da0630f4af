// Host runtime of the C ABI in include/dsm.h: argument validation, the arena
// and chunk layout, the per-context state machine of Algorithm 1, the fp64
// precomputation of the fp32 scalar coefficients, and kernel launches.
// The runtime owns only host memory; every device buffer is the caller's.
#include "dsm.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "dsm_internal.h"

struct dsm_ctx {
    int n = 0, H = 0, n_tensors = 0, base = 0;
    std::vector<int64_t> numel, offsets;
    std::vector<uint8_t> decay;
    int64_t arena_elems = 0;
    std::vector<dsm::Chunk> chunks;  // host copy; the device copy lives in the workspace
    dsm::RepLayout rep{};            // how x_rep holds the n replicas
    dsm::StateLayout ml{};           // how g_rep, s1_rep and s2_rep hold theirs
    dsm::XcdMaps maps{};             // XCD map of each kernel kind for this layout
    std::vector<int32_t> chunk0;     // first chunk of each tensor, then n_chunks (host copy)
    dsm_buffers buf{};
    dsm::Chunk* d_chunks = nullptr;
    dsm::BoundWords bound{};         // workspace words of the randomized sign's bound
    hipStream_t stream = nullptr;
    std::vector<int> local_count;  // local steps per worker since the last synchronisation
    std::vector<uint8_t> stale;    // replica not yet reset to x after a global step
                                   // without broadcast: its next local step reads x
    bool bounds_valid = false;     // the last global step was randomized
    int static_device = -1;        // device whose static scratch the context holds (dsm_init_static)
    std::string last_error;
};

namespace {

thread_local std::string g_last_error;

// Which devices' static scratch a live context made by dsm_init_static holds.
std::mutex g_static_mu;
bool g_static_busy[dsm::kMaxDevices] = {};

constexpr int64_t kMaxNumel = int64_t(1) << 34;
// A launch has n_chunks * kSplit work-groups of kBlockThreads threads per
// grid row, and a grid dimension holds fewer than 2^32 threads.
constexpr int64_t kMaxChunks = ((int64_t(1) << 32) / dsm::kBlockThreads - 1) / dsm::kSplit;

dsm_status fail(dsm_ctx* ctx, dsm_status st, const char* fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(msg, sizeof msg, fmt, ap);
    va_end(ap);
    g_last_error = msg;
    if (ctx) ctx->last_error = msg;
    return st;
}

dsm_status hip_fail(dsm_ctx* ctx, const char* what, hipError_t e) {
    return fail(ctx, DSM_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), static_cast<int>(e));
}

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }

bool finite_in(float v, float lo, float hi) { return std::isfinite(v) && v >= lo && v <= hi; }

struct Layout {
    std::vector<int64_t> offsets;
    int64_t arena_elems = 0;
    int64_t n_chunks = 0;
    int64_t chunk_bytes = 0;
    int64_t bounds_off = 0;
    int64_t chunk0_off = 0;
    int64_t piece_max_off = 0;
    int64_t workspace_bytes = 0;
};

dsm_status check_problem(const dsm_problem* p) {
    if (!p) return fail(nullptr, DSM_ERR_INVALID_ARG, "problem is NULL");
    if (p->n_workers < 1 || p->n_workers > dsm::kMaxWorkers)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "n_workers must be in [1, %d], got %d",
                    dsm::kMaxWorkers, p->n_workers);
    if (p->local_steps < 1)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "local_steps must be >= 1, got %d", p->local_steps);
    if (p->n_tensors < 0)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "n_tensors must be >= 0, got %d", p->n_tensors);
    if (p->base != DSM_BASE_ADAMW && p->base != DSM_BASE_SGD_MOMENTUM)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "unknown base optimizer %d", p->base);
    if (p->replica_layout != DSM_REPLICAS_CONTIGUOUS && p->replica_layout != DSM_REPLICAS_BLOCKED &&
        p->replica_layout != DSM_REPLICAS_STATE_BLOCKED)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "unknown replica layout %d", p->replica_layout);
    if (p->n_tensors > 0 && !p->numel)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "numel is NULL");
    for (int i = 0; i < p->n_tensors; ++i) {
        if (p->numel[i] < 0 || p->numel[i] >= kMaxNumel)
            return fail(nullptr, DSM_ERR_INVALID_ARG, "numel[%d] = %lld outside [0, 2^34)", i,
                        static_cast<long long>(p->numel[i]));
    }
    return DSM_OK;
}

// Tensors back to back, each starting at a multiple of 64 elements (of the
// blocked alignment, with the arena a whole number of the layout's blocks,
// when the replicas are blocked).  The workspace holds, each part at a 256-byte boundary: the chunk table
// (kChunkElems elements per chunk, never crossing a tensor); the per-tensor
// bound words; the first chunk of each tensor (n_tensors + 1 words); and one
// piece-maximum word per work-group piece (n_chunks * kSplit), level one of
// the bound.
dsm_status make_layout(const dsm_problem* p, Layout* L, std::vector<dsm::Chunk>* chunks,
                       std::vector<int32_t>* chunk0 = nullptr) {
    const bool blocked = p->replica_layout != DSM_REPLICAS_CONTIGUOUS;
    const int64_t align = blocked ? dsm::kBlockedTensorAlign : dsm::kTensorAlign;
    const int64_t block = p->replica_layout == DSM_REPLICAS_BLOCKED ? dsm::kRepBlockElems
                                                                     : dsm::kStateBlockElems;
    L->offsets.resize(p->n_tensors);
    int64_t off = 0, n_chunks = 0;
    for (int i = 0; i < p->n_tensors; ++i) {
        L->offsets[i] = off;
        off += round_up(p->numel[i], align);
        n_chunks += (p->numel[i] + dsm::kChunkElems - 1) / dsm::kChunkElems;
    }
    if (blocked) off = round_up(off, block);
    if (n_chunks > kMaxChunks)
        return fail(nullptr, DSM_ERR_UNSUPPORTED, "problem needs %lld chunks, limit %lld",
                    static_cast<long long>(n_chunks), static_cast<long long>(kMaxChunks));
    L->arena_elems = off;
    L->n_chunks = n_chunks;
    L->chunk_bytes = round_up(n_chunks * static_cast<int64_t>(sizeof(dsm::Chunk)), 256);
    L->bounds_off = L->chunk_bytes;
    L->chunk0_off = L->bounds_off + round_up(int64_t(p->n_tensors) * 4, 256);
    L->piece_max_off =
        L->chunk0_off + (p->n_tensors > 0 ? round_up((int64_t(p->n_tensors) + 1) * 4, 256) : 0);
    L->workspace_bytes = L->piece_max_off + round_up(n_chunks * dsm::kSplit * 4, 256);
    if (chunk0) {
        chunk0->assign(p->n_tensors + 1, 0);
        int64_t k = 0;
        for (int i = 0; i < p->n_tensors; ++i) {
            (*chunk0)[i] = static_cast<int32_t>(k);
            k += (p->numel[i] + dsm::kChunkElems - 1) / dsm::kChunkElems;
        }
        (*chunk0)[p->n_tensors] = static_cast<int32_t>(k);
    }
    if (chunks) {
        chunks->clear();
        chunks->reserve(n_chunks);
        for (int i = 0; i < p->n_tensors; ++i) {
            const uint32_t dec = p->decay ? (p->decay[i] ? 1u : 0u) : 1u;
            for (int64_t j = 0; j < p->numel[i]; j += dsm::kChunkElems) {
                dsm::Chunk c{};
                c.off = L->offsets[i] + j;
                c.j0 = j;
                c.len = static_cast<int32_t>(std::min<int64_t>(dsm::kChunkElems, p->numel[i] - j));
                c.tensor = static_cast<uint32_t>(i);
                c.decay = dec;
                chunks->push_back(c);
            }
        }
    }
    return DSM_OK;
}

// beta^s in fp64 by binary exponentiation (square and multiply, lowest bit
// of s first): O(log s) operations for any s and beta.
double beta_power(double beta, int64_t s) {
    double result = 1.0, base = beta;
    for (uint64_t e = static_cast<uint64_t>(s); e > 0; e >>= 1) {
        if (e & 1u) result *= base;
        base *= base;
    }
    return result;
}

dsm_status check_ctx(dsm_ctx* ctx) {
    if (!ctx) return fail(nullptr, DSM_ERR_INVALID_ARG, "context is NULL");
    return DSM_OK;
}

dsm_status check_device(dsm_ctx* ctx) {
    int count = 0;
    hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count == 0)
        return fail(ctx, DSM_ERR_HIP, "no HIP device available (%s)",
                    e == hipSuccess ? "0 devices" : hipGetErrorString(e));
    return DSM_OK;
}

struct LocalCoefs {
    dsm::AdamScalars adam{};
    dsm::SgdScalars sgd{};
};

// Validates the local hyperparameters and forms the fp32 coefficients of one
// local step (fp64, rounded once).
dsm_status local_coefs(dsm_ctx* ctx, const dsm_local_hparams* hp, int64_t step, LocalCoefs* out) {
    if (!hp) return fail(ctx, DSM_ERR_INVALID_ARG, "local hyperparameters are NULL");
    if (!(std::isfinite(hp->lr) && hp->lr > 0.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "lr must be finite and > 0");
    if (!finite_in(hp->beta1, 0.0f, 1.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "beta1 must be in [0, 1]");
    if (ctx->base == DSM_BASE_ADAMW) {
        if (step < 1) return fail(ctx, DSM_ERR_INVALID_ARG, "step must be >= 1, got %lld",
                                  static_cast<long long>(step));
        if (!finite_in(hp->beta2, 0.0f, 1.0f))
            return fail(ctx, DSM_ERR_INVALID_ARG, "beta2 must be in [0, 1]");
        if (!(std::isfinite(hp->eps) && hp->eps >= 0.0f))
            return fail(ctx, DSM_ERR_INVALID_ARG, "eps must be finite and >= 0");
        if (!(std::isfinite(hp->weight_decay) && hp->weight_decay >= 0.0f))
            return fail(ctx, DSM_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
        if (hp->beta1 == 1.0f || hp->beta2 == 1.0f)
            return fail(ctx, DSM_ERR_INVALID_ARG, "AdamW needs beta1, beta2 < 1 (bias correction)");
        const double b1 = hp->beta1, b2 = hp->beta2;
        dsm::AdamScalars& sc = out->adam;
        sc.beta1 = hp->beta1;
        sc.beta2 = hp->beta2;
        sc.one_minus_beta1 = static_cast<float>(1.0 - b1);
        sc.one_minus_beta2 = static_cast<float>(1.0 - b2);
        sc.bc1 = static_cast<float>(1.0 - beta_power(b1, step));
        sc.bc2 = static_cast<float>(1.0 - beta_power(b2, step));
        sc.lr = hp->lr;
        sc.eps = hp->eps;
        sc.wd = hp->weight_decay;
    } else {
        out->sgd = dsm::SgdScalars{hp->beta1, hp->lr};
    }
    return DSM_OK;
}

// Validates the global hyperparameters and forms the fp32 coefficients of
// Eqs. (6)-(8) (fp64, rounded once).
dsm_status global_coefs(dsm_ctx* ctx, int64_t t, const dsm_global_hparams* hp,
                        dsm::GlobalScalars* out) {
    if (!hp) return fail(ctx, DSM_ERR_INVALID_ARG, "global hyperparameters are NULL");
    if (t < 0 || t >= (int64_t(1) << 32))
        return fail(ctx, DSM_ERR_INVALID_ARG, "t must be in [0, 2^32), got %lld", static_cast<long long>(t));
    if (!(std::isfinite(hp->gamma) && hp->gamma > 0.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "gamma must be finite and > 0");
    if (!(std::isfinite(hp->eta) && hp->eta >= 0.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "eta must be finite and >= 0");
    if (!finite_in(hp->beta1, 0.0f, 1.0f) || !finite_in(hp->beta2, 0.0f, 1.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "beta1 and beta2 must be in [0, 1]");
    if (!(std::isfinite(hp->lambda) && hp->lambda >= 0.0f))
        return fail(ctx, DSM_ERR_INVALID_ARG, "lambda must be finite and >= 0");
    if (hp->mode != DSM_SIGN_DET && hp->mode != DSM_SIGN_RAND_FLIP && hp->mode != DSM_SIGN_RAND_ZERO)
        return fail(ctx, DSM_ERR_INVALID_ARG, "unknown sign mode %d", hp->mode);
    if (hp->mode != DSM_SIGN_DET && ctx->arena_elems > 0 && !ctx->buf.u_scratch)
        return fail(ctx, DSM_ERR_INVALID_ARG, "the randomized sign needs buffers.u_scratch");
    if (hp->rule < DSM_RULE_SIGN_MOMENTUM || hp->rule > DSM_RULE_GLOBAL_ADAMW)
        return fail(ctx, DSM_ERR_INVALID_ARG, "unknown global rule %d", hp->rule);
    if (hp->rule != DSM_RULE_SIGN_MOMENTUM && hp->mode != DSM_SIGN_DET)
        return fail(ctx, DSM_ERR_INVALID_ARG,
                    "the randomized sign applies to the sign-momentum rule only");
    if (hp->rule == DSM_RULE_GLOBAL_ADAMW) {
        if (ctx->arena_elems > 0 && !ctx->buf.v)
            return fail(ctx, DSM_ERR_INVALID_ARG, "Global AdamW needs buffers.v");
        if (!(std::isfinite(hp->eps) && hp->eps >= 0.0f))
            return fail(ctx, DSM_ERR_INVALID_ARG, "eps must be finite and >= 0");
        if (hp->beta1 == 1.0f || hp->beta2 == 1.0f)
            return fail(ctx, DSM_ERR_INVALID_ARG, "Global AdamW needs beta1, beta2 < 1");
    }
    dsm::GlobalScalars& sc = *out;
    const double gamma = hp->gamma;
    sc.beta1 = hp->beta1;
    sc.beta2 = hp->beta2;
    sc.c1 = static_cast<float>((1.0 - static_cast<double>(hp->beta1)) / gamma);
    sc.c2 = static_cast<float>((1.0 - static_cast<double>(hp->beta2)) / gamma);
    sc.step = static_cast<float>(static_cast<double>(hp->eta) * gamma);
    sc.lam = hp->lambda;
    sc.n = ctx->n;
    sc.n_pow2 = (ctx->n & (ctx->n - 1)) == 0 ? 1 : 0;
    sc.inv_n = static_cast<float>(1.0 / ctx->n);
    sc.n_f = static_cast<float>(ctx->n);
    sc.key0 = static_cast<uint32_t>(hp->seed & 0xFFFFFFFFu);
    sc.key1 = static_cast<uint32_t>(hp->seed >> 32);
    sc.t = static_cast<uint32_t>(t);
    sc.mode = hp->mode;
    sc.rule = hp->rule;
    sc.inv_gamma = static_cast<float>(1.0 / gamma);
    sc.one_minus_beta1 = static_cast<float>(1.0 - static_cast<double>(hp->beta1));
    sc.one_minus_beta2 = static_cast<float>(1.0 - static_cast<double>(hp->beta2));
    sc.bc1 = static_cast<float>(1.0 - beta_power(hp->beta1, t + 1));
    sc.bc2 = static_cast<float>(1.0 - beta_power(hp->beta2, t + 1));
    sc.eta = hp->eta;
    sc.eps = hp->eps;
    return DSM_OK;
}

hipError_t launch_local(dsm_ctx* ctx, const LocalCoefs& lc, const float* src, dsm::RepLayout sl,
                        int w0, int nw) {
    const int64_t n_chunks = static_cast<int64_t>(ctx->chunks.size());
    if (ctx->base == DSM_BASE_ADAMW)
        return dsm::launch_local_adamw(ctx->d_chunks, n_chunks, ctx->buf.x_rep, ctx->rep, src, sl,
                                       ctx->buf.g_rep, ctx->buf.s1_rep, ctx->buf.s2_rep,
                                       ctx->ml, w0, nw, lc.adam, ctx->maps.local, ctx->stream);
    return dsm::launch_local_sgdm(ctx->d_chunks, n_chunks, ctx->buf.x_rep, ctx->rep, src, sl,
                                  ctx->buf.g_rep, ctx->buf.s1_rep, ctx->ml, w0, nw, lc.sgd,
                                  ctx->maps.local, ctx->stream);
}

// After a global step: the round's local counts restart; without broadcast
// every replica is stale until its worker's next local step.
void end_round(dsm_ctx* ctx, bool broadcast, bool randomized) {
    for (int i = 0; i < ctx->n; ++i) {
        ctx->local_count[i] = 0;
        ctx->stale[i] = broadcast ? 0 : 1;
    }
    ctx->bounds_valid = randomized;
}

}  // namespace

extern "C" {

dsm_status dsm_layout(const dsm_problem* problem, int64_t* arena_elems, int64_t* tensor_offsets,
                      int64_t* workspace_bytes) {
    dsm_status st = check_problem(problem);
    if (st != DSM_OK) return st;
    Layout L;
    st = make_layout(problem, &L, nullptr);
    if (st != DSM_OK) return st;
    if (arena_elems) *arena_elems = L.arena_elems;
    if (tensor_offsets && problem->n_tensors > 0)
        std::memcpy(tensor_offsets, L.offsets.data(), sizeof(int64_t) * problem->n_tensors);
    if (workspace_bytes) *workspace_bytes = L.workspace_bytes;
    return DSM_OK;
}

}  // extern "C"

namespace {

// dsm_init and dsm_init_static.  With use_static, the context's workspace and
// the randomized sign's u staging are the static scratch of the current
// device (the caller's workspace, workspace_bytes and u_scratch are ignored),
// and the device is marked as held until dsm_destroy.
dsm_status init_context(const dsm_problem* problem, const dsm_buffers* caller, dsm_ctx** out,
                        bool use_static) {
    if (!out) return fail(nullptr, DSM_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    dsm_status st = check_problem(problem);
    if (st != DSM_OK) return st;
    if (!caller) return fail(nullptr, DSM_ERR_INVALID_ARG, "buffers is NULL");
    Layout L;
    std::vector<dsm::Chunk> chunks;
    std::vector<int32_t> chunk0;
    st = make_layout(problem, &L, &chunks, &chunk0);
    if (st != DSM_OK) return st;
    const bool adamw = problem->base == DSM_BASE_ADAMW;
    dsm_buffers staged = *caller;
    const dsm_buffers* b = &staged;
    int device = -1;
    std::unique_lock<std::mutex> hold;
    if (use_static) {
        const int64_t u_off = round_up(L.workspace_bytes, 256);
        const int64_t need = u_off + round_up(L.arena_elems * 4, 256);
        if (need > dsm::kStaticScratchBytes)
            return fail(nullptr, DSM_ERR_INVALID_ARG,
                        "problem needs %lld bytes of scratch (workspace and u staging); the "
                        "static scratch of dsm_init_static holds %lld",
                        static_cast<long long>(need),
                        static_cast<long long>(dsm::kStaticScratchBytes));
        st = check_device(nullptr);
        if (st != DSM_OK) return st;
        hipError_t e = hipGetDevice(&device);
        if (e != hipSuccess) return hip_fail(nullptr, "querying the current device", e);
        if (device < 0 || device >= dsm::kMaxDevices)
            return fail(nullptr, DSM_ERR_UNSUPPORTED, "device %d beyond the static scratch table",
                        device);
        hold = std::unique_lock<std::mutex>(g_static_mu);
        if (g_static_busy[device])
            return fail(nullptr, DSM_ERR_STATE,
                        "a context made by dsm_init_static is alive on device %d; destroy it first",
                        device);
        void* scratch = nullptr;
        e = dsm::static_scratch(&scratch);
        if (e != hipSuccess) return hip_fail(nullptr, "finding the static scratch", e);
        staged.workspace = scratch;
        staged.workspace_bytes = L.workspace_bytes;
        staged.u_scratch = reinterpret_cast<float*>(static_cast<char*>(scratch) + u_off);
    }
    if (L.arena_elems > 0) {
        struct {
            const void* p;
            const char* name;
            bool required;
        } ptrs[] = {{b->x, "x", true},           {b->m, "m", true},
                    {b->x_rep, "x_rep", true},   {b->g_rep, "g_rep", true},
                    {b->s1_rep, "s1_rep", true}, {b->s2_rep, "s2_rep", adamw},
                    {b->u_scratch, "u_scratch", false}, {b->v, "v", false}};
        for (const auto& q : ptrs) {
            if (q.required && !q.p)
                return fail(nullptr, DSM_ERR_INVALID_ARG, "buffer %s is NULL", q.name);
            if (q.p && !aligned256(q.p))
                return fail(nullptr, DSM_ERR_INVALID_ARG, "buffer %s is not 256-byte aligned", q.name);
        }
    }
    // How the per-worker buffers hold their n copies.
    dsm::RepLayout rep = dsm::contiguous_copies(L.arena_elems);
    dsm::StateLayout ml{rep, rep, rep};
    if (problem->replica_layout == DSM_REPLICAS_BLOCKED) {
        rep = dsm::blocked_copies(problem->n_workers);
    } else if (problem->replica_layout == DSM_REPLICAS_STATE_BLOCKED) {
        const int nb = adamw ? 4 : 3;
        rep = dsm::state_blocked_copies(problem->n_workers, nb);
        ml = dsm::StateLayout{rep, rep, rep};
        // One allocation: g_rep, s1_rep (and s2_rep) start 1, 2 (and 3) times
        // n blocks after x_rep.
        const int64_t gap = int64_t(problem->n_workers) * dsm::kStateBlockElems;
        if (L.arena_elems > 0 &&
            (b->g_rep != b->x_rep + gap || b->s1_rep != b->x_rep + 2 * gap ||
             (adamw && b->s2_rep != b->x_rep + 3 * gap)))
            return fail(nullptr, DSM_ERR_INVALID_ARG,
                        "state-blocked layout: g_rep, s1_rep%s must start %lld, %lld%s floats "
                        "after x_rep, in one allocation of %d * n * d_pad floats",
                        adamw ? " and s2_rep" : "", static_cast<long long>(gap),
                        static_cast<long long>(2 * gap), adamw ? " and 3x that" : "", nb);
    }
    if (L.workspace_bytes > 0) {
        if (!b->workspace) return fail(nullptr, DSM_ERR_INVALID_ARG, "workspace is NULL");
        if (!aligned256(b->workspace))
            return fail(nullptr, DSM_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
        if (b->workspace_bytes < L.workspace_bytes)
            return fail(nullptr, DSM_ERR_INVALID_ARG, "workspace has %lld bytes, needs %lld",
                        static_cast<long long>(b->workspace_bytes),
                        static_cast<long long>(L.workspace_bytes));
    }
    st = check_device(nullptr);
    if (st != DSM_OK) return st;

    dsm_ctx* ctx = new (std::nothrow) dsm_ctx();
    if (!ctx) return fail(nullptr, DSM_ERR_INVALID_ARG, "out of host memory");
    ctx->n = problem->n_workers;
    ctx->H = problem->local_steps;
    ctx->n_tensors = problem->n_tensors;
    ctx->base = problem->base;
    ctx->numel.assign(problem->numel, problem->numel + problem->n_tensors);
    ctx->decay.resize(problem->n_tensors);
    for (int i = 0; i < problem->n_tensors; ++i)
        ctx->decay[i] = problem->decay ? (problem->decay[i] ? 1 : 0) : 1;
    ctx->offsets = L.offsets;
    ctx->arena_elems = L.arena_elems;
    ctx->rep = rep;
    ctx->ml = ml;
    ctx->maps = dsm::kMapsByLayout[problem->replica_layout];
    ctx->chunks = std::move(chunks);
    ctx->chunk0 = std::move(chunk0);
    ctx->buf = *b;
    ctx->stream = static_cast<hipStream_t>(b->stream);
    char* ws = static_cast<char*>(b->workspace);
    ctx->d_chunks = reinterpret_cast<dsm::Chunk*>(ws);
    ctx->bound.bits = reinterpret_cast<uint32_t*>(ws + L.bounds_off);
    ctx->bound.chunk0 = reinterpret_cast<const int32_t*>(ws + L.chunk0_off);
    ctx->bound.piece_max = reinterpret_cast<uint32_t*>(ws + L.piece_max_off);
    ctx->local_count.assign(ctx->n, 0);
    ctx->stale.assign(ctx->n, 0);

    if (ctx->n_tensors > 0) {
        hipError_t e = hipMemcpyAsync(const_cast<int32_t*>(ctx->bound.chunk0), ctx->chunk0.data(),
                                      ctx->chunk0.size() * sizeof(int32_t),
                                      hipMemcpyHostToDevice, ctx->stream);
        if (e != hipSuccess) {
            dsm_status r = hip_fail(nullptr, "uploading the tensor chunk index", e);
            delete ctx;
            return r;
        }
    }
    if (!ctx->chunks.empty()) {
        hipError_t e = hipMemcpyAsync(ctx->d_chunks, ctx->chunks.data(),
                                      ctx->chunks.size() * sizeof(dsm::Chunk),
                                      hipMemcpyHostToDevice, ctx->stream);
        if (e != hipSuccess) {
            dsm_status r = hip_fail(nullptr, "uploading the chunk table", e);
            delete ctx;
            return r;
        }
        e = dsm::launch_init(ctx->d_chunks, static_cast<int64_t>(ctx->chunks.size()), b->x, b->m,
                             b->v, b->x_rep, ctx->rep, b->s1_rep, adamw ? b->s2_rep : nullptr,
                             ctx->ml, ctx->n, ctx->maps.copy, ctx->stream);
        if (e != hipSuccess) {
            dsm_status r = hip_fail(nullptr, "launching the initialisation kernel", e);
            delete ctx;
            return r;
        }
    }
    if (use_static) {
        ctx->static_device = device;
        g_static_busy[device] = true;
    }
    *out = ctx;
    return DSM_OK;
}

}  // namespace

extern "C" {

dsm_status dsm_init(const dsm_problem* problem, const dsm_buffers* buffers, dsm_ctx** out) {
    return init_context(problem, buffers, out, false);
}

dsm_status dsm_init_static(const dsm_problem* problem, const dsm_buffers* buffers,
                           dsm_ctx** out) {
    return init_context(problem, buffers, out, true);
}

dsm_status dsm_local_step(dsm_ctx* ctx, int32_t worker, int64_t step, const dsm_local_hparams* hp) {
    dsm_status st = check_ctx(ctx);
    if (st != DSM_OK) return st;
    if (worker < -1 || worker >= ctx->n)
        return fail(ctx, DSM_ERR_INVALID_ARG, "worker must be -1 or in [0, %d), got %d", ctx->n, worker);
    LocalCoefs lc;
    st = local_coefs(ctx, hp, step, &lc);
    if (st != DSM_OK) return st;
    const int w0 = worker < 0 ? 0 : worker;
    const int nw = worker < 0 ? ctx->n : 1;
    for (int i = w0; i < w0 + nw; ++i) {
        if (ctx->local_count[i] >= ctx->H)
            return fail(ctx, DSM_ERR_STATE,
                        "worker %d already took H = %d local steps this round; take the global step",
                        i, ctx->H);
    }
    // Workers whose replica is stale read the global model (the
    // synchronisation step folded into their first local step).  When every
    // worker steps and every replica is stale, one launch reads x once for all
    // of them; otherwise one launch per run of consecutive workers with the
    // same source.
    bool all_stale = worker < 0 && ctx->n > 1;
    for (int i = 0; i < ctx->n && all_stale; ++i) all_stale = ctx->stale[i] != 0;
    if (all_stale) {
        hipError_t e = dsm::launch_local_from_x(
            ctx->d_chunks, static_cast<int64_t>(ctx->chunks.size()), ctx->buf.x, ctx->buf.x_rep,
            ctx->rep, ctx->buf.g_rep, ctx->buf.s1_rep, ctx->buf.s2_rep, ctx->ml, ctx->n,
            ctx->base == DSM_BASE_ADAMW, lc.adam, lc.sgd, ctx->maps.from_x, ctx->stream);
        if (e != hipSuccess) return hip_fail(ctx, "launching the local step", e);
    }
    for (int a = w0; a < w0 + nw && !all_stale;) {
        int b = a + 1;
        while (b < w0 + nw && ctx->stale[b] == ctx->stale[a]) ++b;
        const bool from_x = ctx->stale[a] != 0;
        const float* src = from_x ? ctx->buf.x : ctx->buf.x_rep;
        const dsm::RepLayout sl = from_x ? dsm::single_copy() : ctx->rep;
        hipError_t e = launch_local(ctx, lc, src, sl, a, b - a);
        if (e != hipSuccess) return hip_fail(ctx, "launching the local step", e);
        a = b;
    }
    for (int i = w0; i < w0 + nw; ++i) {
        ctx->local_count[i] += 1;
        ctx->stale[i] = 0;
    }
    return DSM_OK;
}

dsm_status dsm_global_step(dsm_ctx* ctx, int64_t t, const dsm_global_hparams* hp, int32_t broadcast) {
    dsm_status st = check_ctx(ctx);
    if (st != DSM_OK) return st;
    dsm::GlobalScalars sc{};
    st = global_coefs(ctx, t, hp, &sc);
    if (st != DSM_OK) return st;
    for (int i = 0; i < ctx->n; ++i) {
        if (ctx->local_count[i] != ctx->H)
            return fail(ctx, DSM_ERR_STATE,
                        "worker %d took %d of H = %d local steps; the global step needs all H",
                        i, ctx->local_count[i], ctx->H);
    }
    const bool randomized = hp->mode != DSM_SIGN_DET;
    const int64_t n_chunks = static_cast<int64_t>(ctx->chunks.size());
    hipError_t e;
    if (!randomized) {
        e = dsm::launch_global_det(ctx->d_chunks, n_chunks, ctx->buf.x, ctx->buf.m, ctx->buf.v,
                                   ctx->buf.x_rep, ctx->rep, sc, broadcast != 0, ctx->maps.global,
                                   ctx->stream);
    } else {
        e = dsm::launch_global_rand(ctx->d_chunks, n_chunks, ctx->n_tensors, ctx->buf.x, ctx->buf.m,
                                    ctx->buf.x_rep, ctx->rep, ctx->buf.u_scratch, ctx->bound, sc,
                                    broadcast != 0, ctx->maps.global, ctx->stream);
    }
    if (e != hipSuccess) return hip_fail(ctx, "launching the global step", e);
    end_round(ctx, broadcast != 0, randomized);
    return DSM_OK;
}

dsm_status dsm_round_end(dsm_ctx* ctx, int64_t step, const dsm_local_hparams* local_hp, int64_t t,
                         const dsm_global_hparams* global_hp, int32_t broadcast) {
    dsm_status st = check_ctx(ctx);
    if (st != DSM_OK) return st;
    LocalCoefs lc;
    st = local_coefs(ctx, local_hp, step, &lc);
    if (st != DSM_OK) return st;
    dsm::GlobalScalars gs{};
    st = global_coefs(ctx, t, global_hp, &gs);
    if (st != DSM_OK) return st;
    if (global_hp->rule != DSM_RULE_SIGN_MOMENTUM)
        return fail(ctx, DSM_ERR_UNSUPPORTED,
                    "dsm_round_end fuses the sign-momentum rule only; use dsm_local_step and "
                    "dsm_global_step for the variants");
    for (int i = 0; i < ctx->n; ++i) {
        if (ctx->local_count[i] != ctx->H - 1)
            return fail(ctx, DSM_ERR_STATE,
                        "worker %d took %d local steps; dsm_round_end takes step H = %d and needs "
                        "H - 1 taken", i, ctx->local_count[i], ctx->H);
    }
    // With H - 1 >= 1 steps taken every replica is fresh; with H = 1 the
    // replicas are all stale or all fresh (no local step since the last
    // global step or synchronisation).
    const bool from_x = ctx->stale[0] != 0;
    dsm::RoundEndArgs a{};
    a.x = ctx->buf.x;
    a.m = ctx->buf.m;
    a.x_rep = ctx->buf.x_rep;
    a.rl = ctx->rep;
    a.x_src = from_x ? ctx->buf.x : ctx->buf.x_rep;
    a.sl = from_x ? dsm::single_copy() : ctx->rep;
    a.g_rep = ctx->buf.g_rep;
    a.s1 = ctx->buf.s1_rep;
    a.s2 = ctx->buf.s2_rep;
    a.u = ctx->buf.u_scratch;
    a.bound = ctx->bound;
    a.ml = ctx->ml;
    a.map = ctx->maps.round_end;
    a.map_pass2 = ctx->maps.global;
    a.as = lc.adam;
    a.ss = lc.sgd;
    a.gs = gs;
    const bool randomized = global_hp->mode != DSM_SIGN_DET;
    hipError_t e = dsm::launch_round_end(ctx->d_chunks, static_cast<int64_t>(ctx->chunks.size()),
                                         ctx->n_tensors, ctx->base == DSM_BASE_ADAMW, a,
                                         broadcast != 0, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, "launching the fused round end", e);
    end_round(ctx, broadcast != 0, randomized);
    return DSM_OK;
}

dsm_status dsm_sync(dsm_ctx* ctx) {
    dsm_status st = check_ctx(ctx);
    if (st != DSM_OK) return st;
    hipError_t e = dsm::launch_broadcast(ctx->d_chunks, static_cast<int64_t>(ctx->chunks.size()),
                                         ctx->buf.x, ctx->buf.x_rep, ctx->rep, ctx->n,
                                         ctx->maps.copy, ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, "launching the synchronisation", e);
    for (int i = 0; i < ctx->n; ++i) {
        ctx->local_count[i] = 0;
        ctx->stale[i] = 0;
    }
    return DSM_OK;
}

dsm_status dsm_read_bounds(dsm_ctx* ctx, float* host_B, int32_t capacity) {
    dsm_status st = check_ctx(ctx);
    if (st != DSM_OK) return st;
    if (!ctx->bounds_valid)
        return fail(ctx, DSM_ERR_STATE, "the last global step did not use the randomized sign");
    if (ctx->n_tensors == 0) return DSM_OK;
    if (!host_B) return fail(ctx, DSM_ERR_INVALID_ARG, "host_B is NULL");
    if (capacity < ctx->n_tensors)
        return fail(ctx, DSM_ERR_INVALID_ARG, "host_B holds %d floats, the problem has %d tensors",
                    capacity, ctx->n_tensors);
    hipError_t e = hipMemcpyAsync(host_B, ctx->bound.bits, sizeof(uint32_t) * ctx->n_tensors,
                                  hipMemcpyDeviceToHost, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, "reading the bounds", e);
    return DSM_OK;
}

dsm_status dsm_test_philox(uint64_t seed, uint32_t tensor, int64_t t, int64_t q0, int64_t count,
                           uint32_t* dev_out, void* stream) {
    if (!dev_out) return fail(nullptr, DSM_ERR_INVALID_ARG, "dev_out is NULL");
    if (count < 0 || q0 < 0 || q0 + count > (int64_t(1) << 32))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "need count >= 0, q0 >= 0, q0 + count <= 2^32");
    if (count > (int64_t(1) << 30))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "count must be <= 2^30");
    if (t < 0 || t >= (int64_t(1) << 32))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "t must be in [0, 2^32)");
    if ((reinterpret_cast<uintptr_t>(dev_out) & 3u) != 0)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "dev_out is not 4-byte aligned");
    dsm_status st = check_device(nullptr);
    if (st != DSM_OK) return st;
    hipError_t e = dsm::launch_test_philox(static_cast<uint32_t>(seed & 0xFFFFFFFFu),
                                           static_cast<uint32_t>(seed >> 32), tensor,
                                           static_cast<uint32_t>(t), static_cast<uint32_t>(q0),
                                           count, dev_out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(nullptr, "launching the Philox test kernel", e);
    return DSM_OK;
}

#if DSM_UNROLL == 1 && DSM_ITERS == 1 && DSM_BLOCK_THREADS == 256
static_assert(dsm::kPieceElems == DSM_PIECE_ELEMS, "dsm.h's piece size is the default build's");
#endif

dsm_status dsm_test_stream(int32_t kind, float* dev_buf, int64_t n_elems, uint32_t* dev_words,
                           uint32_t pattern, void* stream) {
    if (kind != DSM_STREAM_READ && kind != DSM_STREAM_WRITE)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "kind must be DSM_STREAM_READ or DSM_STREAM_WRITE");
    // A build with other work-group shape knobs has another piece size than
    // the one dsm.h promises for the word array.
    if (dsm::kPieceElems != DSM_PIECE_ELEMS)
        return fail(nullptr, DSM_ERR_UNSUPPORTED, "this build's piece is %lld elements, not %d",
                    static_cast<long long>(dsm::kPieceElems), DSM_PIECE_ELEMS);
    if (n_elems < 0 || n_elems % dsm::kPieceElems != 0)
        return fail(nullptr, DSM_ERR_INVALID_ARG, "n_elems must be a non-negative multiple of %lld",
                    static_cast<long long>(dsm::kPieceElems));
    const int64_t n_pieces = n_elems / dsm::kPieceElems;
    if (n_pieces * dsm::kBlockThreads >= (int64_t(1) << 32))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "n_elems exceeds one grid dimension (%lld pieces)",
                    static_cast<long long>(n_pieces));
    if (n_elems > 0 && (!dev_buf || !aligned256(dev_buf)))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "dev_buf is NULL or not 256-byte aligned");
    if (kind == DSM_STREAM_READ && n_elems > 0 &&
        (!dev_words || (reinterpret_cast<uintptr_t>(dev_words) & 3u) != 0))
        return fail(nullptr, DSM_ERR_INVALID_ARG, "dev_words is NULL or not 4-byte aligned");
    dsm_status st = check_device(nullptr);
    if (st != DSM_OK) return st;
    hipError_t e = dsm::launch_test_stream(kind, dev_buf, n_pieces, dev_words, pattern,
                                           static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(nullptr, "launching the streaming test kernel", e);
    return DSM_OK;
}

dsm_status dsm_destroy(dsm_ctx* ctx) {
    if (!ctx) return DSM_OK;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (ctx->static_device >= 0) {
        // The context's work has drained (or the stream failed); the next
        // dsm_init_static on this device may reuse the scratch.
        std::lock_guard<std::mutex> lock(g_static_mu);
        g_static_busy[ctx->static_device] = false;
    }
    delete ctx;
    if (e != hipSuccess) return hip_fail(nullptr, "synchronising the stream at destroy", e);
    return DSM_OK;
}

const char* dsm_last_error(const dsm_ctx* ctx) {
    return ctx ? ctx->last_error.c_str() : g_last_error.c_str();
}

}  // extern "C"
