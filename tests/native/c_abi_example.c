/*
 * The C ABI of include/dsm.h used from plain C (no Python, no torch): device
 * buffers from hipMalloc, one fused round with the lazy broadcast, then one
 * split round with broadcast, then checks on the host:
 *   - every replica equals x bit for bit after the broadcast (Algorithm 1
 *     synchronisation step);
 *   - with lambda = 0, x moved by exactly eta * gamma per element on which the
 *     sign of u is +-1, and not at all where it is 0 (Eq. (7));
 * then one round with the randomized sign of Eq. (10), whose per-tensor
 * bounds must equal max |u| of the staged u, and whose steps must be 0 or
 * eta * gamma in the direction of sign(u);
 *   - every error path returns a status and a message.
 * All of it twice: with contiguous replicas (the ABI default), and with the
 * replicas and their optimizer state in 16 KiB blocks of one allocation
 * (DSM_REPLICAS_STATE_BLOCKED), whose gradients go in with a pitched copy.
 * Prints "c abi example ok" and exits 0, or names the failed check and
 * exits 1.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dsm.h"

#define HIP_OK(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess) {                                                       \
            printf("HIP error %d at line %d\n", (int)e_, __LINE__);                   \
            return 1;                                                                 \
        }                                                                             \
    } while (0)
#define DSM_OK_(call)                                                                 \
    do {                                                                              \
        dsm_status s_ = (call);                                                       \
        if (s_ != DSM_OK) {                                                           \
            printf("dsm status %d at line %d: %s\n", (int)s_, __LINE__, dsm_last_error(NULL)); \
            return 1;                                                                 \
        }                                                                             \
    } while (0)

static uint32_t lcg(uint32_t* s) {
    *s = *s * 1664525u + 1013904223u;
    return *s;
}

/* Where copy i of element e of per-worker buffer j (0 x_rep, 1 g_rep, 2 s1, 3 s2)
   sits: in that buffer's own allocation at i * d_pad + e, or, with the state
   blocked, in the one allocation of 4 * n * d_pad floats, block e / 4096 of
   4 * n copies of 4096 elements each. */
#define STATE_BLOCK 4096
static size_t slot(int layout, int64_t arena, int n, int j, int i, int64_t e) {
    if (layout == DSM_REPLICAS_STATE_BLOCKED)
        return (size_t)((e / STATE_BLOCK) * (4 * n * STATE_BLOCK) + (j * n + i) * STATE_BLOCK +
                        e % STATE_BLOCK);
    return (size_t)(i * arena + e);
}

/* Random gradients for every worker, in the buffer's own layout. */
static int upload_grads(int layout, float* g_rep, float* hg, int64_t arena, int n, uint32_t* seed,
                        hipStream_t st) {
    const size_t count = (size_t)arena * (size_t)n;
    for (size_t j = 0; j < count; ++j) hg[j] = ((float)(lcg(seed) >> 8) / 16777216.0f - 0.5f) * 0.02f;
    if (layout == DSM_REPLICAS_STATE_BLOCKED) {
        /* Block b holds the n gradient copies contiguously, n * 4096 floats in,
           one block length (4 * n * 4096 floats) after block b - 1. */
        const size_t width = (size_t)n * STATE_BLOCK * sizeof(float);
        HIP_OK(hipMemcpy2DAsync(g_rep, 4 * width, hg, width, width, (size_t)(arena / STATE_BLOCK),
                                hipMemcpyHostToDevice, st));
    } else {
        HIP_OK(hipMemcpyAsync(g_rep, hg, count * sizeof(float), hipMemcpyHostToDevice, st));
    }
    HIP_OK(hipStreamSynchronize(st));
    return 0;
}

static int run(int layout) {
    const int64_t numel[3] = {5, 1000, 16385};
    const uint8_t decay[3] = {0, 1, 1};
    const int n = 3, H = 2;
    dsm_problem prob = {n, H, 3, DSM_BASE_ADAMW, numel, decay, layout};
    int64_t arena = 0, offs[3], ws = 0;
    DSM_OK_(dsm_layout(&prob, &arena, offs, &ws));
    const int blocked = layout == DSM_REPLICAS_STATE_BLOCKED;
    if (blocked && arena % STATE_BLOCK != 0) {
        printf("state-blocked arena of %lld elements is not whole blocks\n", (long long)arena);
        return 1;
    }

    const size_t one = (size_t)arena * sizeof(float), many = one * (size_t)n;
    /* The host copy of the replicas covers the one allocation when blocked. */
    const size_t reps = blocked ? 4 * many : many;
    float *x, *m, *x_rep, *g_rep, *s1, *s2, *u;
    void* work;
    HIP_OK(hipMalloc((void**)&x, one));
    HIP_OK(hipMalloc((void**)&m, one));
    if (blocked) {
        HIP_OK(hipMalloc((void**)&x_rep, 4 * many));
        g_rep = x_rep + (size_t)n * STATE_BLOCK;
        s1 = x_rep + 2 * (size_t)n * STATE_BLOCK;
        s2 = x_rep + 3 * (size_t)n * STATE_BLOCK;
    } else {
        HIP_OK(hipMalloc((void**)&x_rep, many));
        HIP_OK(hipMalloc((void**)&g_rep, many));
        HIP_OK(hipMalloc((void**)&s1, many));
        HIP_OK(hipMalloc((void**)&s2, many));
    }
    HIP_OK(hipMalloc((void**)&u, one));
    HIP_OK(hipMalloc(&work, (size_t)ws));

    float* hx = (float*)malloc(one);
    float* hx1 = (float*)malloc(one);
    float* hg = (float*)malloc(many);
    float* hr = (float*)malloc(reps);
    float* hu = (float*)malloc(one);
    if (!hx || !hx1 || !hg || !hr || !hu) return 1;
    uint32_t seed = 12345u;
    for (int64_t j = 0; j < arena; ++j) hx[j] = ((float)(lcg(&seed) >> 8) / 16777216.0f - 0.5f) * 0.04f;
    HIP_OK(hipMemcpy(x, hx, one, hipMemcpyHostToDevice));

    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));
    dsm_buffers buf = {x, m, x_rep, g_rep, s1, s2, u, work, ws, st, NULL};
    dsm_ctx* ctx = NULL;
    DSM_OK_(dsm_init(&prob, &buf, &ctx));

    dsm_local_hparams lh = {1e-3f, 0.9f, 0.95f, 1e-8f, 0.1f};
    dsm_global_hparams gh = {1e-3f, 0.8f, 0.95f, 0.98f, 0.0f, DSM_SIGN_DET, 0, DSM_RULE_SIGN_MOMENTUM, 1e-8f};
    int64_t s = 0;
    for (int t = 0; t < 2; ++t) {
        for (int k = 0; k < H; ++k) {
            if (upload_grads(layout, g_rep, hg, arena, n, &seed, st)) return 1;
            ++s;
            if (t == 0 && k == H - 1)
                DSM_OK_(dsm_round_end(ctx, s, &lh, t, &gh, 0));       /* fused, lazy */
            else
                DSM_OK_(dsm_local_step(ctx, -1, s, &lh));
        }
        if (t == 1) {
            HIP_OK(hipStreamSynchronize(st));
            HIP_OK(hipMemcpy(hx, x, one, hipMemcpyDeviceToHost));   /* x before the step */
            DSM_OK_(dsm_global_step(ctx, t, &gh, 1));              /* split, broadcast */
        }
    }
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipMemcpy(hx1, x, one, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hr, x_rep, reps, hipMemcpyDeviceToHost));

    /* Replicas equal x on every tensor element. */
    for (int i = 0; i < n; ++i)
        for (int p = 0; p < 3; ++p)
            for (int64_t j = 0; j < numel[p]; ++j)
                if (memcmp(hr + slot(layout, arena, n, 0, i, offs[p] + j), hx1 + offs[p] + j,
                           sizeof(float)) != 0) {
                    printf("replica %d differs from x on tensor %d\n", i, p);
                    return 1;
                }
    /* lambda = 0: x - x_new is +-eta*gamma rounded, or 0. */
    const float step = (float)((double)0.8f * (double)1e-3f);   /* as the runtime forms eta * gamma */
    int64_t moved = 0;
    for (int p = 0; p < 3; ++p)
        for (int64_t j = 0; j < numel[p]; ++j) {
            const float a = hx[offs[p] + j], b = hx1[offs[p] + j];
            const float d = a - b;
            const float plus = a - step, minus = a + step;
            if (!(b == a || b == plus || b == minus)) {
                printf("tensor %d element %lld moved by %g, not +-%g\n", p, (long long)j, d, step);
                return 1;
            }
            moved += (b != a);
        }
    if (moved == 0) {
        printf("no element moved\n");
        return 1;
    }

    float no_bounds[3];
    if (dsm_read_bounds(ctx, no_bounds, 3) != DSM_ERR_STATE) {
        printf("bounds of a deterministic step were not refused\n");
        return 1;
    }

    /* Round t = 2 with the randomized sign of Eq. (10), split, with broadcast. */
    for (int k = 0; k < H; ++k) {
        if (upload_grads(layout, g_rep, hg, arena, n, &seed, st)) return 1;
        DSM_OK_(dsm_local_step(ctx, -1, ++s, &lh));
    }
    dsm_global_hparams gz = gh;
    gz.mode = DSM_SIGN_RAND_ZERO;
    gz.seed = 0x0123456789ABCDEFull;
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipMemcpy(hx, x, one, hipMemcpyDeviceToHost));
    DSM_OK_(dsm_global_step(ctx, 2, &gz, 1));
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipMemcpy(hx1, x, one, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hu, u, one, hipMemcpyDeviceToHost));
    float bound[3] = {-1.0f, -1.0f, -1.0f};
    DSM_OK_(dsm_read_bounds(ctx, bound, 3));
    int64_t kept = 0;
    for (int p = 0; p < 3; ++p) {
        float want = 0.0f;
        for (int64_t j = 0; j < numel[p]; ++j) {
            const float a = fabsf(hu[offs[p] + j]);
            if (a > want) want = a;
        }
        if (memcmp(&want, &bound[p], sizeof want) != 0) {
            printf("tensor %d: bound %g, max |u| %g\n", p, bound[p], want);
            return 1;
        }
        for (int64_t j = 0; j < numel[p]; ++j) {
            /* Eq. (10) keeps sign(u) or gives 0: x moves by eta*gamma against
               sign(u), or not at all (lambda = 0). */
            const float a = hx[offs[p] + j], b = hx1[offs[p] + j], uu = hu[offs[p] + j];
            const float moved = uu > 0.0f ? a - step : (uu < 0.0f ? a + step : a);
            if (!(b == a || b == moved)) {
                printf("randomized step: tensor %d element %lld moved to %g from %g\n", p,
                       (long long)j, b, a);
                return 1;
            }
            kept += (b != a);
        }
    }
    if (kept == 0) {
        printf("the randomized sign kept no sign\n");
        return 1;
    }

    /* Error paths return a status and a message. */
    if (dsm_global_step(ctx, 2, &gh, 1) != DSM_ERR_STATE || strlen(dsm_last_error(ctx)) == 0) {
        printf("global step before H local steps was not refused\n");
        return 1;
    }
    float small_bounds[2];
    if (dsm_read_bounds(ctx, small_bounds, 2) != DSM_ERR_INVALID_ARG) {
        printf("a bound array shorter than n_tensors was not refused\n");
        return 1;
    }
    DSM_OK_(dsm_destroy(ctx));
    HIP_OK(hipFree(x)); HIP_OK(hipFree(m)); HIP_OK(hipFree(x_rep));
    if (!blocked) {
        HIP_OK(hipFree(g_rep)); HIP_OK(hipFree(s1)); HIP_OK(hipFree(s2));
    }
    HIP_OK(hipFree(u)); HIP_OK(hipFree(work));
    HIP_OK(hipStreamDestroy(st));
    free(hx); free(hx1); free(hg); free(hr); free(hu);
    printf("%s replicas: %lld elements moved by one sign step, %lld signs kept by the "
           "randomized step\n", blocked ? "state-blocked" : "contiguous", (long long)moved,
           (long long)kept);
    return 0;
}

int main(void) {
    if (run(DSM_REPLICAS_CONTIGUOUS) || run(DSM_REPLICAS_STATE_BLOCKED)) return 1;
    printf("c abi example ok\n");
    return 0;
}
