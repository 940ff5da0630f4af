// gfx950 kernels of distributed sign momentum with local steps
// (arXiv 2411.17866, Algorithm 1).
//
// Every kernel streams fp32 arenas: each work-group takes one piece of one
// chunk of one tensor (Chunk; by default 256 threads x one float4 = 1024
// elements), each thread moves 128-bit (float4) groups with nontemporal loads
// and stores, consecutive threads touch consecutive 16-byte groups, and every
// element is read and written once per pass.  Nothing here is a
// dense contraction, so there is no MFMA; the bound is HBM bandwidth.
//
// Arithmetic: fp32, one IEEE round-to-nearest operation per written
// operation, in the order the formulas are written; no contraction into FMA
// (-ffp-contract=off and the pragma below), correctly rounded division and
// square root, denormals kept.
#include <hip/hip_runtime.h>

#include <mutex>

#include "dsm_internal.h"
#include "philox_device.h"

#pragma clang fp contract(off)

namespace dsm {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// Whether the streams use nontemporal loads and stores, and how far the
// fused round end unrolls its worker loop (build-time knobs).
#ifndef DSM_NT
#define DSM_NT 1
#endif
#ifndef DSM_ROUND_END_UNROLL
#define DSM_ROUND_END_UNROLL 0
#endif

__device__ __forceinline__ f4 ntload(const f4* p) {
#if DSM_NT
    return __builtin_nontemporal_load(p);
#else
    return *p;
#endif
}
__device__ __forceinline__ void ntstore(f4 v, f4* p) {
#if DSM_NT
    __builtin_nontemporal_store(v, p);
#else
    *p = v;
#endif
}

// Stores the first k (1..3) lanes of v: the ragged end of a tensor.
__device__ __forceinline__ void store_head(f4 v, float* p, int k) {
    p[0] = v.x;
    if (k > 1) p[1] = v.y;
    if (k > 2) p[2] = v.z;
}

// Stores v at p: the whole group when its four lanes are inside the chunk
// (valid >= 4), else only the valid lanes.
__device__ __forceinline__ void store_vec(f4 v, f4* p, int valid) {
    if (valid >= 4)
        ntstore(v, p);
    else
        store_head(v, reinterpret_cast<float*>(p), valid);
}

// Where copy i of a replica buffer keeps arena element e (RepLayout):
// (e >> shift) * block_stride + i * copy_stride + (e & (2^shift - 1)).
// Contiguous copies use shift 62 (the block term vanishes) and copy_stride =
// d_pad; 64 KiB blocks interleaved by copy use shift 14, block_stride =
// n * 16384 and copy_stride = 16384; "every copy is x" uses shift 62 and
// copy_stride 0.  A piece never crosses a block, so one base per piece and
// copy serves every thread of the work-group.
__device__ __forceinline__ int64_t rep_index(const RepLayout& L, int64_t i, int64_t e) {
    const int64_t mask = (int64_t(1) << L.shift) - 1;
    return (e >> L.shift) * L.block_stride + i * L.copy_stride + (e & mask);
}

// The piece of a chunk this work-group processes: work item w (below) takes
// piece w % kSplit of chunk w / kSplit, kPieceVec float4 groups from group
// (w % kSplit) * kPieceVec of the chunk on (fewer at the chunk's end).
// Work-groups are short-lived and handle one piece each, so the addresses in
// flight form compact fronts that sweep the arena.
struct Piece {
    Chunk c;
    uint32_t wi;     // piece index: chunk wi / kSplit, piece wi % kSplit of it
    int nq;          // float4 groups in the piece (0 past the chunk's end)
    int valid0;      // lanes of the chunk from the piece's first group on
    int64_t e0;      // arena element of the piece's first group
    uint32_t j4;     // in-tensor index of the first group, divided by 4
};

constexpr uint32_t kXcds = 8;  // MI355X: work-groups go to its 8 XCDs round-robin

// Work item of this work-group.  MAP 0: the work-group index itself (XCD k
// takes piece k mod 8 of every chunk).  1: XCD k takes the k-th eighth of the
// grid row, in order.  2: XCD k takes whole chunks (chunk 8r + k in group r).
// Modes 1 and 2 are bijections on a prefix of the row and the identity on the
// rest.
template <int MAP>
__device__ __forceinline__ uint32_t work_index() {
    const uint32_t b = blockIdx.x;
    if constexpr (MAP == 1) {
        const uint32_t per = gridDim.x / kXcds;
        if (b >= per * kXcds) return b;
        return (b % kXcds) * per + b / kXcds;
    } else if constexpr (MAP == 2) {
        const uint32_t group = kXcds * kSplit;
        if (b >= (gridDim.x / group) * group) return b;
        const uint32_t r = b / kXcds, x = b % kXcds;
        return (r / kSplit) * group + x * kSplit + r % kSplit;
    } else {
        return b;
    }
}

// The map is a launch argument (the runtime picks it per kernel kind and
// replica layout) and uniform over the grid, so the branch is scalar.
__device__ __forceinline__ uint32_t work_index(int map) {
    if (map == 1) return work_index<1>();
    if (map == 2) return work_index<2>();
    return work_index<0>();
}

__device__ __forceinline__ Piece piece_at(const Chunk* __restrict__ chunks, uint32_t wi) {
    Piece pc;
    pc.wi = wi;
    pc.c = chunks[wi / kSplit];
    const int nvec = (pc.c.len + 3) >> 2;
    const int q_lo = static_cast<int>(wi % kSplit) * kPieceVec;
    pc.nq = max(0, min(nvec, q_lo + kPieceVec) - q_lo);
    pc.valid0 = pc.c.len - 4 * q_lo;
    pc.e0 = pc.c.off + 4 * static_cast<int64_t>(q_lo);
    pc.j4 = static_cast<uint32_t>(pc.c.j0 >> 2) + static_cast<uint32_t>(q_lo);
    return pc;
}

__device__ __forceinline__ Piece piece_of(const Chunk* __restrict__ chunks, int map) {
    return piece_at(chunks, work_index(map & 3));
}

// The piece and worker of a local-step work-group.  Without kInterleaveWorkers
// in the map the grid is (pieces, workers) and runs worker by worker; with it
// the grid is one row of pieces x workers, worker fastest, so consecutive
// work-groups take the same piece of successive workers.
__device__ __forceinline__ Piece local_piece(const Chunk* __restrict__ chunks, int map, int worker0,
                                             int n_workers, int64_t& w) {
    if (map & kInterleaveWorkers) {
        const uint32_t f = work_index(map & 3);
        w = worker0 + static_cast<int64_t>(f % static_cast<uint32_t>(n_workers));
        return piece_at(chunks, f / static_cast<uint32_t>(n_workers));
    }
    w = worker0 + static_cast<int64_t>(blockIdx.y);
    return piece_at(chunks, work_index(map & 3));
}

// ---------------------------------------------------------------- AdamW

// Correctly rounded square root (the build asks for correctly rounded fp32
// division and square root).
__device__ __forceinline__ f4 sqrt_rn(f4 a) {
    return f4{__builtin_sqrtf(a.x), __builtin_sqrtf(a.y), __builtin_sqrtf(a.z), __builtin_sqrtf(a.w)};
}

// Algorithm 2 on four elements (lane-wise); x, m, v updated in place.
__device__ __forceinline__ void adamw4(f4& x, f4 g, f4& m, f4& v, float lam, const AdamScalars& s) {
    const f4 m1 = s.beta1 * m;
    const f4 m2 = s.one_minus_beta1 * g;
    m = m1 + m2;
    const f4 gg = g * g;
    const f4 v1 = s.beta2 * v;
    const f4 v2 = s.one_minus_beta2 * gg;
    v = v1 + v2;
    const f4 m_hat = m / s.bc1;
    const f4 v_hat = v / s.bc2;
    const f4 den = sqrt_rn(v_hat) + s.eps;
    const f4 r = m_hat / den;
    const f4 wx = lam * x;
    const f4 d = r + wx;
    const f4 st = s.lr * d;
    x = x - st;
}

// Worker w reads its step's starting point at x_src + rep_index(sl, w, e)
// (its own replica, or with a zero copy stride the global model x when the
// replicas are stale after a global step without broadcast) and writes the
// result to its replica, x_rep + rep_index(rl, w, e); its gradient and
// moments sit at rep_index(ml.g / ml.s1 / ml.s2, w, e) of their buffers.  The two may be the
// same memory, so neither pointer is __restrict__; each thread loads every
// stream of its group before it stores.
__global__ __launch_bounds__(kBlockThreads) void k_local_adamw(
    const Chunk* __restrict__ chunks, int map, float* x_rep, RepLayout rl, const float* x_src,
    RepLayout sl, const float* __restrict__ g_rep, float* __restrict__ s1,
    float* __restrict__ s2, StateLayout ml, int worker0, int n_workers, AdamScalars sc) {
    int64_t w;
    const Piece pc = local_piece(chunks, map, worker0, n_workers, w);
    f4* xp = reinterpret_cast<f4*>(x_rep + rep_index(rl, w, pc.e0));
    const f4* xs = reinterpret_cast<const f4*>(x_src + rep_index(sl, w, pc.e0));
    const f4* __restrict__ gp = reinterpret_cast<const f4*>(g_rep + rep_index(ml.g, w, pc.e0));
    f4* __restrict__ mp = reinterpret_cast<f4*>(s1 + rep_index(ml.s1, w, pc.e0));
    f4* __restrict__ vp = reinterpret_cast<f4*>(s2 + rep_index(ml.s2, w, pc.e0));
    const float lam = pc.c.decay ? sc.wd : 0.0f;
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], gv[kUnroll], mv[kUnroll], vv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xs + q);
                gv[k] = ntload(gp + q);
                mv[k] = ntload(mp + q);
                vv[k] = ntload(vp + q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                const int valid = pc.valid0 - 4 * q;
                adamw4(xv[k], gv[k], mv[k], vv[k], lam, sc);
                store_vec(xv[k], xp + q, valid);
                store_vec(mv[k], mp + q, valid);
                store_vec(vv[k], vp + q, valid);
            }
        }
    }
}

// ---------------------------------------------------------------- SGD + momentum

// Algorithm 3 on four elements (lane-wise).
__device__ __forceinline__ void sgdm4(f4& x, f4 g, f4& m, const SgdScalars& s) {
    const f4 m1 = s.mu * m;
    m = m1 + g;
    const f4 st = s.lr * m;
    x = x - st;
}

__global__ __launch_bounds__(kBlockThreads) void k_local_sgdm(
    const Chunk* __restrict__ chunks, int map, float* x_rep, RepLayout rl, const float* x_src,
    RepLayout sl, const float* __restrict__ g_rep, float* __restrict__ s1, StateLayout ml,
    int worker0, int n_workers, SgdScalars sc) {
    int64_t w;
    const Piece pc = local_piece(chunks, map, worker0, n_workers, w);
    f4* xp = reinterpret_cast<f4*>(x_rep + rep_index(rl, w, pc.e0));
    const f4* xs = reinterpret_cast<const f4*>(x_src + rep_index(sl, w, pc.e0));
    const f4* __restrict__ gp = reinterpret_cast<const f4*>(g_rep + rep_index(ml.g, w, pc.e0));
    f4* __restrict__ mp = reinterpret_cast<f4*>(s1 + rep_index(ml.s1, w, pc.e0));
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], gv[kUnroll], mv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xs + q);
                gv[k] = ntload(gp + q);
                mv[k] = ntload(mp + q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                const int valid = pc.valid0 - 4 * q;
                sgdm4(xv[k], gv[k], mv[k], sc);
                store_vec(xv[k], xp + q, valid);
                store_vec(mv[k], mp + q, valid);
            }
        }
    }
}

// ---------------------------------------------------------------- global step

// sign with sign(+-0) = +0 and sign(NaN) = NaN.
__device__ __forceinline__ float sign_of(float u) {
    return u > 0.0f ? 1.0f : (u < 0.0f ? -1.0f : (u == u ? 0.0f : u));
}

// Worker sum of (x - x_i) over the n replicas of group q of the piece that
// starts at arena element e0, in worker order, divided by n.  N > 0:
// compile-time worker count (a power of two, so the division is the exact
// multiplication by 1/n); N == 0: runtime count.
template <int N>
__device__ __forceinline__ f4 worker_mean_diff(f4 xv, const float* __restrict__ x_rep,
                                               const RepLayout& rl, int64_t e0, int q,
                                               const GlobalScalars& s) {
    if constexpr (N > 0) {
        f4 r[N];
#pragma unroll
        for (int i = 0; i < N; ++i)
            r[i] = ntload(reinterpret_cast<const f4*>(x_rep + rep_index(rl, i, e0)) + q);
        f4 acc = xv - r[0];
#pragma unroll
        for (int i = 1; i < N; ++i) acc = acc + (xv - r[i]);
        return acc * s.inv_n;
    } else {
        f4 acc = xv - ntload(reinterpret_cast<const f4*>(x_rep + rep_index(rl, 0, e0)) + q);
        for (int i = 1; i < s.n; ++i)
            acc = acc + (xv - ntload(reinterpret_cast<const f4*>(x_rep + rep_index(rl, i, e0)) + q));
        if (s.n_pow2) return acc * s.inv_n;
        return acc / s.n_f;
    }
}

__device__ __forceinline__ f4 sign4(f4 u) {
    return f4{sign_of(u.x), sign_of(u.y), sign_of(u.z), sign_of(u.w)};
}

// Eqs. (6) and (8) from the old m, lane-wise; returns u, updates m.
__device__ __forceinline__ f4 momentum4(f4& m, f4 delta, const GlobalScalars& s) {
    const f4 u1 = s.beta1 * m;
    const f4 u2 = s.c1 * delta;
    const f4 u = u1 + u2;
    const f4 m1 = s.beta2 * m;
    const f4 m2 = s.c2 * delta;
    m = m1 + m2;
    return u;
}

// Eq. (7) with the applied sign S, lane-wise.
__device__ __forceinline__ f4 model4(f4 x, f4 S, float lam, const GlobalScalars& s) {
    const f4 wx = lam * x;
    const f4 a = S + wx;
    const f4 st = s.step * a;
    return x - st;
}

// Global-step rules (dsm_global_rule).
constexpr int kRuleSignMomentum = 0;  // Eqs. (6)-(8)
constexpr int kRuleLookahead = 1;     // Section 4.1: x - eta gamma (u + lambda x)
constexpr int kRuleSignedSlowMo = 2;  // Section 4.1: sign on the averaged difference
constexpr int kRuleGlobalAdamW = 3;   // Algorithm 7

// Algorithm 7 on four elements: AdamW on the pseudo-gradient
// g = (1/gamma) delta; m and v updated in place; returns the new x.
__device__ __forceinline__ f4 global_adamw4(f4 x, f4 delta, f4& m, f4& v, float lam,
                                           const GlobalScalars& s) {
    const f4 g = s.inv_gamma * delta;
    const f4 m1 = s.beta1 * m;
    const f4 m2 = s.one_minus_beta1 * g;
    m = m1 + m2;
    const f4 gg = g * g;
    const f4 v1 = s.beta2 * v;
    const f4 v2 = s.one_minus_beta2 * gg;
    v = v1 + v2;
    const f4 m_hat = m / s.bc1;
    const f4 v_hat = v / s.bc2;
    const f4 den = sqrt_rn(v_hat) + s.eps;
    const f4 r = m_hat / den;
    const f4 wx = lam * x;
    const f4 d = r + wx;
    const f4 st = s.eta * d;
    return x - st;
}

template <int N, int RULE, bool BCAST>
__global__ __launch_bounds__(kBlockThreads) void k_global_det(
    const Chunk* __restrict__ chunks, int map, float* __restrict__ x, float* __restrict__ m,
    float* __restrict__ v, float* __restrict__ x_rep, RepLayout rl, GlobalScalars sc) {
    const Piece pc = piece_of(chunks, map);
    const int n = N > 0 ? N : sc.n;
    f4* __restrict__ xp = reinterpret_cast<f4*>(x + pc.e0);
    f4* __restrict__ mp = reinterpret_cast<f4*>(m + pc.e0);
    f4* __restrict__ vp = reinterpret_cast<f4*>(v + pc.e0);
    const float lam = pc.c.decay ? sc.lam : 0.0f;
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], mv[kUnroll], vv[kUnroll], dv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xp + q);
                mv[k] = ntload(mp + q);
                if (RULE == kRuleGlobalAdamW) vv[k] = ntload(vp + q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) dv[k] = worker_mean_diff<N>(xv[k], x_rep, rl, pc.e0, q, sc);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                const int valid = pc.valid0 - 4 * q;
                f4 xn;
                if constexpr (RULE == kRuleSignMomentum) {
                    const f4 u = momentum4(mv[k], dv[k], sc);
                    xn = model4(xv[k], sign4(u), lam, sc);
                } else if constexpr (RULE == kRuleLookahead) {
                    const f4 u = momentum4(mv[k], dv[k], sc);
                    xn = model4(xv[k], u, lam, sc);
                } else if constexpr (RULE == kRuleSignedSlowMo) {
                    // u from the old m and the sign of the difference; m by Eq. (8).
                    const f4 u1 = sc.beta1 * mv[k];
                    const f4 u2 = sc.c1 * sign4(dv[k]);
                    const f4 u = u1 + u2;
                    const f4 m1 = sc.beta2 * mv[k];
                    const f4 m2 = sc.c2 * dv[k];
                    mv[k] = m1 + m2;
                    xn = model4(xv[k], u, lam, sc);
                } else {
                    xn = global_adamw4(xv[k], dv[k], mv[k], vv[k], lam, sc);
                    store_vec(vv[k], vp + q, valid);
                }
                store_vec(xn, xp + q, valid);
                store_vec(mv[k], mp + q, valid);
                if (BCAST) {
                    for (int i = 0; i < n; ++i)
                        store_vec(xn, reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0)) + q,
                                  valid);
                }
            }
        }
    }
}

// Largest of the values of a work-group of THREADS threads, valid in thread
// 0.  wave_max holds THREADS / 64 words of LDS.
template <int THREADS>
__device__ __forceinline__ uint32_t block_max(uint32_t bits, uint32_t* wave_max) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(bits, off, 64);
        bits = o > bits ? o : bits;
    }
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (lane == 0) wave_max[wave] = bits;
    __syncthreads();
    uint32_t b = wave_max[0];
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < THREADS / 64; ++w) b = wave_max[w] > b ? wave_max[w] : b;
    }
    return b;
}

// The tensor bound B_p = max |u| is reduced in two levels, with plain loads
// and stores and no atomics.  Level one: each work-group stores the largest
// |u| of its piece, as a bit pattern, in the piece's own slot (for
// non-negative IEEE floats the unsigned order of the bit patterns is the
// numeric order).  Level two is k_bound_reduce.
__device__ __forceinline__ void store_piece_max(uint32_t bits, uint32_t* wave_max,
                                                uint32_t* slot) {
    const uint32_t b = block_max<kBlockThreads>(bits, wave_max);
    if (threadIdx.x == 0) *slot = b;
}

// Randomized sign, pass 1: the all-reduce difference, u_{t+1} (staged to u)
// and m_{t+1} (Eqs. (6), (8)), and the tensor bound B_p = max |u|.
template <int N>
__global__ __launch_bounds__(kBlockThreads) void k_global_rand_pass1(
    const Chunk* __restrict__ chunks, int map, const float* __restrict__ x, float* __restrict__ m,
    const float* __restrict__ x_rep, RepLayout rl, float* __restrict__ u_out,
    uint32_t* __restrict__ piece_max, GlobalScalars sc) {
    const Piece pc = piece_of(chunks, map);
    const f4* __restrict__ xp = reinterpret_cast<const f4*>(x + pc.e0);
    f4* __restrict__ mp = reinterpret_cast<f4*>(m + pc.e0);
    f4* __restrict__ up = reinterpret_cast<f4*>(u_out + pc.e0);
    __shared__ uint32_t wave_max[kBlockThreads / 64];
    uint32_t maxbits = 0;
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], mv[kUnroll], dv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xp + q);
                mv[k] = ntload(mp + q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) dv[k] = worker_mean_diff<N>(xv[k], x_rep, rl, pc.e0, q, sc);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                const int valid = pc.valid0 - 4 * q;  // lanes inside the tensor
                const f4 uv = momentum4(mv[k], dv[k], sc);
                store_vec(uv, up + q, valid);
                store_vec(mv[k], mp + q, valid);
                uint32_t b = __float_as_uint(fabsf(uv.x));
                if (valid > 1) b = max(b, __float_as_uint(fabsf(uv.y)));
                if (valid > 2) b = max(b, __float_as_uint(fabsf(uv.z)));
                if (valid > 3) b = max(b, __float_as_uint(fabsf(uv.w)));
                maxbits = max(maxbits, b);
            }
        }
    }
    store_piece_max(maxbits, wave_max, piece_max + pc.wi);
}

// Level two of the tensor bound: work-group p takes the piece maxima of
// tensor p (slots chunk0[p] * kSplit up to chunk0[p + 1] * kSplit, the pieces
// of its chunks) and stores their largest in bound_bits[p]; an empty tensor
// has no slots and gets 0.
constexpr int kReduceThreads = 1024;
__global__ __launch_bounds__(kReduceThreads) void k_bound_reduce(
    const uint32_t* __restrict__ piece_max, const int32_t* __restrict__ chunk0,
    uint32_t* __restrict__ bound_bits) {
    __shared__ uint32_t wave_max[kReduceThreads / 64];
    const int p = blockIdx.x;
    const int64_t lo = static_cast<int64_t>(chunk0[p]) * kSplit;
    const int64_t hi = static_cast<int64_t>(chunk0[p + 1]) * kSplit;
    uint32_t b = 0;
    if constexpr (kSplit % 4 == 0) {
        // lo is a multiple of 4 slots, and the slots start 256-byte aligned.
        const uint4* __restrict__ v = reinterpret_cast<const uint4*>(piece_max + lo);
        const int64_t nv = (hi - lo) / 4;
#pragma unroll 4
        for (int64_t i = threadIdx.x; i < nv; i += kReduceThreads) {
            const uint4 w = v[i];
            b = max(b, max(max(w.x, w.y), max(w.z, w.w)));
        }
    } else {
        for (int64_t i = lo + threadIdx.x; i < hi; i += kReduceThreads) b = max(b, piece_max[i]);
    }
    b = block_max<kReduceThreads>(b, wave_max);
    if (threadIdx.x == 0) bound_bits[p] = b;
}

// S_r(u) of Eq. (9) (MODE 1) or Eq. (10) (MODE 2) for one element, given the
// Philox word w (U = (w >> 8) 2^-24) and the bound B (as double).  "sign(u)
// with probability p" is decided by the exact comparison U < p, evaluated in
// fp64 where both sides are exact: (2k - 2^24) B < |u| 2^24 for Eq. (9),
// k B < |u| 2^24 for Eq. (10).
template <int MODE>
__device__ __forceinline__ float rand_sign(float u, uint32_t w, double B) {
    const float sgn = sign_of(u);
    const double au = static_cast<double>(fabsf(u)) * 16777216.0;
    const int32_t k = static_cast<int32_t>(w >> 8);
    if constexpr (MODE == 1) {
        const double a = static_cast<double>(2 * k - (1 << 24));
        return (a * B < au) ? sgn : 0.0f - sgn;
    } else {
        return (static_cast<double>(k) * B < au) ? sgn : 0.0f;
    }
}

// Randomized sign, pass 2: S_r, Eq. (7) and the synchronisation step.
// Section 3.1 defines S_r only for a finite bound: a tensor whose bound is
// NaN or infinite (it holds a non-finite u) gets S = NaN at every element,
// so its step is NaN rather than a step of a reversed or zero sign.
template <int MODE, bool BCAST>
__global__ __launch_bounds__(kBlockThreads) void k_global_rand_pass2(
    const Chunk* __restrict__ chunks, int map, float* __restrict__ x, float* __restrict__ x_rep,
    RepLayout rl, const float* __restrict__ u_in, const uint32_t* __restrict__ bound_bits,
    GlobalScalars sc) {
    const Piece pc = piece_of(chunks, map);
    const Chunk& c = pc.c;
    f4* __restrict__ xp = reinterpret_cast<f4*>(x + pc.e0);
    const f4* __restrict__ up = reinterpret_cast<const f4*>(u_in + pc.e0);
    const float lam = c.decay ? sc.lam : 0.0f;
    const uint32_t bbits = bound_bits[c.tensor];
    const bool bound_finite = bbits < 0x7f800000u;   // B >= 0: below the +inf pattern
    const double B = static_cast<double>(__uint_as_float(bbits));
    const float undefined = __builtin_nanf("");
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], uv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xp + q);
                uv[k] = ntload(up + q);
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                uint32_t w0 = pc.j4 + static_cast<uint32_t>(q), w1 = c.tensor, w2 = sc.t,
                         w3 = kSignStream;
                philox4x32_10(w0, w1, w2, w3, sc.key0, sc.key1);
                f4 S = {rand_sign<MODE>(uv[k].x, w0, B), rand_sign<MODE>(uv[k].y, w1, B),
                        rand_sign<MODE>(uv[k].z, w2, B), rand_sign<MODE>(uv[k].w, w3, B)};
                if (!bound_finite) S = f4{undefined, undefined, undefined, undefined};
                const f4 xn = model4(xv[k], S, lam, sc);
                const int valid = pc.valid0 - 4 * q;
                store_vec(xn, xp + q, valid);
                if (BCAST) {
                    for (int i = 0; i < sc.n; ++i)
                        store_vec(xn, reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0)) + q,
                                  valid);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- local step from x

// Base optimizer of the kernels that take local steps of several workers.
constexpr int kBaseAdamW = 0;
constexpr int kBaseSgd = 1;

// Local step of every worker when every replica is stale (after a global
// step without broadcast): each worker's x_{t+1,0} is the global model, so
// the work-group reads x once and takes the step of all n workers on it,
// writing each replica, instead of one pass per worker that re-reads x.  The
// per-element arithmetic is adamw4 / sgdm4, as in the per-worker kernels.
template <int N, int BASE>
__global__ __launch_bounds__(kBlockThreads) void k_local_from_x(
    const Chunk* __restrict__ chunks, int map, const float* __restrict__ x, float* __restrict__ x_rep,
    RepLayout rl, const float* __restrict__ g_rep, float* __restrict__ s1,
    float* __restrict__ s2, StateLayout ml, int n_rt, AdamScalars as, SgdScalars ss) {
    const Piece pc = piece_of(chunks, map);
    const int n = N > 0 ? N : n_rt;
    const f4* __restrict__ xp = reinterpret_cast<const f4*>(x + pc.e0);
    const float lam = pc.c.decay ? as.wd : 0.0f;
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) xv[k] = ntload(xp + q);
        }
#if DSM_ROUND_END_UNROLL == 0
#pragma unroll(N > 0 ? N : 1)
#elif DSM_ROUND_END_UNROLL == 1
#pragma unroll 1
#elif DSM_ROUND_END_UNROLL == 2
#pragma unroll 2
#endif
        for (int i = 0; i < (N > 0 ? N : n); ++i) {
            f4* __restrict__ xr = reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0));
            const f4* __restrict__ gp = reinterpret_cast<const f4*>(g_rep + rep_index(ml.g, i, pc.e0));
            f4* __restrict__ s1p = reinterpret_cast<f4*>(s1 + rep_index(ml.s1, i, pc.e0));
            f4* __restrict__ s2p = reinterpret_cast<f4*>(s2 + rep_index(ml.s2, i, pc.e0));
            f4 gi[kUnroll], mi[kUnroll], vi[kUnroll];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int q = q0 + k * kBlockThreads;
                if (q < pc.nq) {
                    gi[k] = ntload(gp + q);
                    mi[k] = ntload(s1p + q);
                    if (BASE == kBaseAdamW) vi[k] = ntload(s2p + q);
                }
            }
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int q = q0 + k * kBlockThreads;
                if (q < pc.nq) {
                    const int valid = pc.valid0 - 4 * q;
                    f4 xi = xv[k];
                    if (BASE == kBaseAdamW) {
                        adamw4(xi, gi[k], mi[k], vi[k], lam, as);
                        store_vec(vi[k], s2p + q, valid);
                    } else {
                        sgdm4(xi, gi[k], mi[k], ss);
                    }
                    store_vec(xi, xr + q, valid);
                    store_vec(mi[k], s1p + q, valid);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- fused round end

// The last local step of every worker (Algorithm 2 or 3, Eq. (4)) fused with
// the global step (all-reduce, Eqs. (6)-(8)): each worker's step-H replica
// value stays in registers and is folded into the worker-order sum
// sum_i (x - x_i) as it is produced, so the replicas are neither stored after
// step H nor read back.  Per element the operations and their order are those
// of k_local_* followed by k_global_det / k_global_rand_pass1, so the results
// are bit-identical.  KIND: 0 deterministic sign, 1 deterministic sign with
// broadcast, 2 randomized pass 1 (u, m and the bound; pass 2 follows).

template <int N, int BASE, int KIND>
__global__ __launch_bounds__(kBlockThreads) void k_round_end(
    const Chunk* __restrict__ chunks, int map, float* x, float* __restrict__ m, float* x_rep,
    RepLayout rl, const float* x_src, RepLayout sl, const float* __restrict__ g_rep,
    float* __restrict__ s1, float* __restrict__ s2, float* __restrict__ u_out,
    uint32_t* __restrict__ piece_max, StateLayout ml, AdamScalars as, SgdScalars ss,
    GlobalScalars gs) {
    // x_src is the replicas or, when they are stale, x itself: it may alias
    // x and x_rep, so none of the three is __restrict__.  Every load of a
    // group precedes its stores.
    __shared__ uint32_t wave_max[kBlockThreads / 64];
    const Piece pc = piece_of(chunks, map);
    const int n = N > 0 ? N : gs.n;
    f4* xp = reinterpret_cast<f4*>(x + pc.e0);
    f4* __restrict__ mp = reinterpret_cast<f4*>(m + pc.e0);
    const float lam_local = pc.c.decay ? as.wd : 0.0f;
    const float lam = pc.c.decay ? gs.lam : 0.0f;
    uint32_t maxbits = 0;
    for (int q0 = threadIdx.x; q0 < pc.nq; q0 += kBlockThreads * kUnroll) {
        f4 xv[kUnroll], mv[kUnroll], acc[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                xv[k] = ntload(xp + q);
                mv[k] = ntload(mp + q);
            }
        }
        // Worker loop: unrolled DSM_ROUND_END_UNROLL workers at a time (0: fully,
        // for a compile-time worker count).  Fully unrolled, every worker's loads
        // are in flight together; that measured faster than the rolled loop's
        // lower register count and higher occupancy.
#if DSM_ROUND_END_UNROLL == 0
#pragma unroll(N > 0 ? N : 1)
#elif DSM_ROUND_END_UNROLL == 1
#pragma unroll 1
#elif DSM_ROUND_END_UNROLL == 2
#pragma unroll 2
#endif
        for (int i = 0; i < (N > 0 ? N : n); ++i) {
            const f4* xs = reinterpret_cast<const f4*>(x_src + rep_index(sl, i, pc.e0));
            const f4* __restrict__ gp = reinterpret_cast<const f4*>(g_rep + rep_index(ml.g, i, pc.e0));
            f4* __restrict__ s1p = reinterpret_cast<f4*>(s1 + rep_index(ml.s1, i, pc.e0));
            f4* __restrict__ s2p = reinterpret_cast<f4*>(s2 + rep_index(ml.s2, i, pc.e0));
            f4 xi[kUnroll], gi[kUnroll], mi[kUnroll], vi[kUnroll];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int q = q0 + k * kBlockThreads;
                if (q < pc.nq) {
                    xi[k] = ntload(xs + q);
                    gi[k] = ntload(gp + q);
                    mi[k] = ntload(s1p + q);
                    if (BASE == kBaseAdamW) vi[k] = ntload(s2p + q);
                }
            }
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int q = q0 + k * kBlockThreads;
                if (q < pc.nq) {
                    const int valid = pc.valid0 - 4 * q;
                    if (BASE == kBaseAdamW) {
                        adamw4(xi[k], gi[k], mi[k], vi[k], lam_local, as);
                        store_vec(vi[k], s2p + q, valid);
                    } else {
                        sgdm4(xi[k], gi[k], mi[k], ss);
                    }
                    store_vec(mi[k], s1p + q, valid);
                    const f4 d = xv[k] - xi[k];
                    acc[k] = (i == 0) ? d : acc[k] + d;
                }
            }
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int q = q0 + k * kBlockThreads;
            if (q < pc.nq) {
                const int valid = pc.valid0 - 4 * q;
                f4 delta;
                if (N > 0 || gs.n_pow2)
                    delta = acc[k] * gs.inv_n;
                else
                    delta = acc[k] / gs.n_f;
                const f4 u = momentum4(mv[k], delta, gs);
                store_vec(mv[k], mp + q, valid);
                if (KIND == 2) {
                    store_vec(u, reinterpret_cast<f4*>(u_out + pc.e0) + q, valid);
                    uint32_t b = __float_as_uint(fabsf(u.x));
                    if (valid > 1) b = max(b, __float_as_uint(fabsf(u.y)));
                    if (valid > 2) b = max(b, __float_as_uint(fabsf(u.z)));
                    if (valid > 3) b = max(b, __float_as_uint(fabsf(u.w)));
                    maxbits = max(maxbits, b);
                } else {
                    const f4 xn = model4(xv[k], sign4(u), lam, gs);
                    store_vec(xn, xp + q, valid);
                    if (KIND == 1) {
                        for (int i = 0; i < n; ++i)
                            store_vec(xn,
                                      reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0)) + q,
                                      valid);
                    }
                }
            }
        }
    }
    if (KIND == 2) store_piece_max(maxbits, wave_max, piece_max + pc.wi);
}

// ---------------------------------------------------------------- sync / init

// Synchronisation step: x_rep[i] <- x for every replica.
__global__ __launch_bounds__(kBlockThreads) void k_broadcast(
    const Chunk* __restrict__ chunks, int map, const float* __restrict__ x, float* __restrict__ x_rep,
    RepLayout rl, int n) {
    const Piece pc = piece_of(chunks, map);
    const f4* __restrict__ xp = reinterpret_cast<const f4*>(x + pc.e0);
    for (int q = threadIdx.x; q < pc.nq; q += kBlockThreads) {
        const f4 v = ntload(xp + q);
        const int valid = pc.valid0 - 4 * q;
        for (int i = 0; i < n; ++i)
            store_vec(v, reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0)) + q, valid);
    }
}

// Algorithm 1 initialisation: m = 0, replicas = x, base state = 0.
__global__ __launch_bounds__(kBlockThreads) void k_init(
    const Chunk* __restrict__ chunks, int map, const float* __restrict__ x, float* __restrict__ m,
    float* __restrict__ v, float* __restrict__ x_rep, RepLayout rl, float* __restrict__ s1,
    float* __restrict__ s2, StateLayout ml, int n) {
    const Piece pc = piece_of(chunks, map);
    const f4* __restrict__ xp = reinterpret_cast<const f4*>(x + pc.e0);
    const f4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int q = threadIdx.x; q < pc.nq; q += kBlockThreads) {
        const f4 xv = ntload(xp + q);
        const int valid = pc.valid0 - 4 * q;
        store_vec(zero, reinterpret_cast<f4*>(m + pc.e0) + q, valid);
        if (v != nullptr) store_vec(zero, reinterpret_cast<f4*>(v + pc.e0) + q, valid);
        for (int i = 0; i < n; ++i) {
            store_vec(xv, reinterpret_cast<f4*>(x_rep + rep_index(rl, i, pc.e0)) + q, valid);
            store_vec(zero, reinterpret_cast<f4*>(s1 + rep_index(ml.s1, i, pc.e0)) + q, valid);
            if (s2 != nullptr)
                store_vec(zero, reinterpret_cast<f4*>(s2 + rep_index(ml.s2, i, pc.e0)) + q, valid);
        }
    }
}

__global__ __launch_bounds__(kBlockThreads) void k_test_philox(uint32_t key0, uint32_t key1,
                                                              uint32_t tensor, uint32_t t,
                                                              uint32_t q0, int64_t count,
                                                              uint32_t* __restrict__ out) {
    const int64_t b = static_cast<int64_t>(blockIdx.x) * kBlockThreads + threadIdx.x;
    if (b >= count) return;
    uint32_t w0 = q0 + static_cast<uint32_t>(b), w1 = tensor, w2 = t, w3 = kSignStream;
    philox4x32_10(w0, w1, w2, w3, key0, key1);
    out[4 * b + 0] = w0;
    out[4 * b + 1] = w1;
    out[4 * b + 2] = w2;
    out[4 * b + 3] = w3;
}

// Streaming diagnostics with the access shape of the kernels above: one
// piece of kPieceVec float4 groups per work-group, XCD map 1, 16-byte
// nontemporal accesses, consecutive lanes on consecutive groups.  The read
// kernel folds its piece into one word (the XOR of its 32-bit patterns) and
// writes only where that word equals `pattern`, so with a pattern no piece
// matches it issues no write at all: even one 4-byte store per piece,
// interleaved with the loads, costs the read stream a measurable share of
// its rate.  The write kernel stores the float with bit pattern `pattern`.
__global__ __launch_bounds__(kBlockThreads) void k_stream_read(const float* __restrict__ buf,
                                                              uint32_t* __restrict__ words,
                                                              uint32_t pattern) {
    __shared__ uint32_t wave_acc[kBlockThreads / 64];
    const uint32_t wi = work_index<1>();
    const f4* __restrict__ p = reinterpret_cast<const f4*>(buf) + static_cast<int64_t>(wi) * kPieceVec;
    uint32_t acc = 0;
    for (int q = threadIdx.x; q < kPieceVec; q += kBlockThreads) {
        const f4 v = ntload(p + q);
        acc ^= __float_as_uint(v.x) ^ __float_as_uint(v.y) ^ __float_as_uint(v.z) ^
               __float_as_uint(v.w);
    }
    for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) wave_acc[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t total = 0;
        for (int k = 0; k < kBlockThreads / 64; ++k) total ^= wave_acc[k];
        if (total == pattern) words[wi] = 1u;
    }
}

__global__ __launch_bounds__(kBlockThreads) void k_stream_write(float* __restrict__ buf,
                                                               uint32_t pattern) {
    const uint32_t wi = work_index<1>();
    f4* __restrict__ p = reinterpret_cast<f4*>(buf) + static_cast<int64_t>(wi) * kPieceVec;
    const float value = __uint_as_float(pattern);
    const f4 v = {value, value, value, value};
    for (int q = threadIdx.x; q < kPieceVec; q += kBlockThreads) ntstore(v, p + q);
}

dim3 chunk_grid(int64_t n_chunks, int n_workers) {
    return dim3(static_cast<unsigned>(n_chunks * kSplit), static_cast<unsigned>(n_workers), 1);
}

// Grid of a local step: one row of pieces x workers when the map interleaves
// the workers, else (pieces, workers).
dim3 local_grid(int64_t n_chunks, int n_workers, int map) {
    if (map & kInterleaveWorkers)
        return dim3(static_cast<unsigned>(n_chunks * kSplit * n_workers), 1, 1);
    return chunk_grid(n_chunks, n_workers);
}

}  // namespace

// ---------------------------------------------------------------- launchers

hipError_t launch_init(const Chunk* chunks, int64_t n_chunks, float* x, float* m, float* v,
                       float* x_rep, RepLayout rl, float* s1, float* s2, StateLayout ml, int n,
                       int map, hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_init, chunk_grid(n_chunks, 1), dim3(kBlockThreads), 0, st, chunks, map, x,
                       m, v, x_rep, rl, s1, s2, ml, n);
    return hipGetLastError();
}

hipError_t launch_local_adamw(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                              const float* x_src, RepLayout sl, const float* g_rep, float* s1,
                              float* s2, StateLayout ml, int worker0, int n_workers,
                              const AdamScalars& sc, int map, hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    map = local_map(n_chunks, n_workers, map);
    hipLaunchKernelGGL(k_local_adamw, local_grid(n_chunks, n_workers, map), dim3(kBlockThreads), 0,
                       st, chunks, map, x_rep, rl, x_src, sl, g_rep, s1, s2, ml, worker0, n_workers,
                       sc);
    return hipGetLastError();
}

hipError_t launch_local_sgdm(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                             const float* x_src, RepLayout sl, const float* g_rep, float* s1,
                             StateLayout ml, int worker0, int n_workers, const SgdScalars& sc,
                             int map, hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    map = local_map(n_chunks, n_workers, map);
    hipLaunchKernelGGL(k_local_sgdm, local_grid(n_chunks, n_workers, map), dim3(kBlockThreads), 0,
                       st, chunks, map, x_rep, rl, x_src, sl, g_rep, s1, ml, worker0, n_workers, sc);
    return hipGetLastError();
}

template <int BASE, int KIND>
static void launch_round_end_n(const Chunk* chunks, int64_t n_chunks, const RoundEndArgs& a,
                               hipStream_t st) {
    const dim3 grid = chunk_grid(n_chunks, 1), block(kBlockThreads);
#define DSM_ROUND_END(NW)                                                                        \
    hipLaunchKernelGGL((k_round_end<NW, BASE, KIND>), grid, block, 0, st, chunks, a.map, a.x, a.m,\
                       a.x_rep, a.rl, a.x_src, a.sl, a.g_rep, a.s1, a.s2, a.u, a.bound.piece_max, \
                       a.ml, a.as, a.ss, a.gs)
    switch (a.gs.n) {
        case 1: DSM_ROUND_END(1); break;
        case 2: DSM_ROUND_END(2); break;
        case 4: DSM_ROUND_END(4); break;
        case 8: DSM_ROUND_END(8); break;
        default: DSM_ROUND_END(0); break;
    }
#undef DSM_ROUND_END
}

template <int BASE>
static void launch_round_end_base(const Chunk* chunks, int64_t n_chunks, const RoundEndArgs& a,
                                  int kind, hipStream_t st) {
    if (kind == 0)
        launch_round_end_n<BASE, 0>(chunks, n_chunks, a, st);
    else if (kind == 1)
        launch_round_end_n<BASE, 1>(chunks, n_chunks, a, st);
    else
        launch_round_end_n<BASE, 2>(chunks, n_chunks, a, st);
}

template <int BASE>
static void launch_local_from_x_n(const Chunk* chunks, int64_t n_chunks, const float* x,
                                  float* x_rep, RepLayout rl, const float* g_rep, float* s1,
                                  float* s2, StateLayout ml, int n, const AdamScalars& as,
                                  const SgdScalars& ss, int map, hipStream_t st) {
    const dim3 grid = chunk_grid(n_chunks, 1), block(kBlockThreads);
#define DSM_LOCAL_FROM_X(NW)                                                                   \
    hipLaunchKernelGGL((k_local_from_x<NW, BASE>), grid, block, 0, st, chunks, map, x, x_rep, rl,\
                       g_rep, s1, s2, ml, n, as, ss)
    switch (n) {
        case 1: DSM_LOCAL_FROM_X(1); break;
        case 2: DSM_LOCAL_FROM_X(2); break;
        case 4: DSM_LOCAL_FROM_X(4); break;
        case 8: DSM_LOCAL_FROM_X(8); break;
        default: DSM_LOCAL_FROM_X(0); break;
    }
#undef DSM_LOCAL_FROM_X
}

hipError_t launch_local_from_x(const Chunk* chunks, int64_t n_chunks, const float* x,
                               float* x_rep, RepLayout rl, const float* g_rep, float* s1,
                               float* s2, StateLayout ml, int n, bool adamw,
                               const AdamScalars& as, const SgdScalars& ss, int map,
                               hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    if (adamw)
        launch_local_from_x_n<kBaseAdamW>(chunks, n_chunks, x, x_rep, rl, g_rep, s1, s2, ml, n,
                                          as, ss, map, st);
    else
        launch_local_from_x_n<kBaseSgd>(chunks, n_chunks, x, x_rep, rl, g_rep, s1, s2, ml, n, as,
                                        ss, map, st);
    return hipGetLastError();
}

// Level two of the tensor bound, after a first pass has stored its piece
// maxima.  Also run with no chunks at all, so that every bound is written.
static void launch_bound_reduce(const BoundWords& bw, int n_tensors, hipStream_t st) {
    hipLaunchKernelGGL(k_bound_reduce, dim3(static_cast<unsigned>(n_tensors)),
                       dim3(kReduceThreads), 0, st, bw.piece_max, bw.chunk0, bw.bits);
}

static void launch_rand_pass2(const Chunk* chunks, int64_t n_chunks, float* x, float* x_rep,
                              RepLayout rl, const float* u, const uint32_t* bits,
                              const GlobalScalars& sc, bool broadcast, int map, hipStream_t st) {
    const dim3 grid = chunk_grid(n_chunks, 1), block(kBlockThreads);
#define DSM_PASS2(MODE, B) \
    hipLaunchKernelGGL((k_global_rand_pass2<MODE, B>), grid, block, 0, st, chunks, map, x, x_rep, rl, u, bits, sc)
    if (sc.mode == 1) {
        if (broadcast) DSM_PASS2(1, true); else DSM_PASS2(1, false);
    } else {
        if (broadcast) DSM_PASS2(2, true); else DSM_PASS2(2, false);
    }
#undef DSM_PASS2
}

hipError_t launch_round_end(const Chunk* chunks, int64_t n_chunks, int n_tensors, bool adamw,
                            const RoundEndArgs& a, bool broadcast, hipStream_t st) {
    const bool randomized = a.gs.mode != 0;
    const int kind = randomized ? 2 : (broadcast ? 1 : 0);
    if (n_chunks > 0) {
        if (adamw)
            launch_round_end_base<kBaseAdamW>(chunks, n_chunks, a, kind, st);
        else
            launch_round_end_base<kBaseSgd>(chunks, n_chunks, a, kind, st);
    }
    if (randomized && n_tensors > 0) launch_bound_reduce(a.bound, n_tensors, st);
    if (randomized && n_chunks > 0)
        launch_rand_pass2(chunks, n_chunks, a.x, a.x_rep, a.rl, a.u, a.bound.bits, a.gs,
                          broadcast, a.map_pass2, st);
    return hipGetLastError();
}

template <int RULE, bool BCAST>
static void launch_global_det_n(const Chunk* chunks, int64_t n_chunks, float* x, float* m,
                                float* v, float* x_rep, RepLayout rl, const GlobalScalars& sc,
                                int map, hipStream_t st) {
    const dim3 grid = chunk_grid(n_chunks, 1), block(kBlockThreads);
#define DSM_GLOBAL_DET(NW)                                                                     \
    hipLaunchKernelGGL((k_global_det<NW, RULE, BCAST>), grid, block, 0, st, chunks, map, x, m, \
                       v, x_rep, rl, sc)
    switch (sc.n) {
        case 1: DSM_GLOBAL_DET(1); break;
        case 2: DSM_GLOBAL_DET(2); break;
        case 4: DSM_GLOBAL_DET(4); break;
        case 8: DSM_GLOBAL_DET(8); break;
        default: DSM_GLOBAL_DET(0); break;
    }
#undef DSM_GLOBAL_DET
}

template <int RULE>
static void launch_global_det_rule(const Chunk* chunks, int64_t n_chunks, float* x, float* m,
                                   float* v, float* x_rep, RepLayout rl, const GlobalScalars& sc,
                                   bool broadcast, int map, hipStream_t st) {
    if (broadcast)
        launch_global_det_n<RULE, true>(chunks, n_chunks, x, m, v, x_rep, rl, sc, map, st);
    else
        launch_global_det_n<RULE, false>(chunks, n_chunks, x, m, v, x_rep, rl, sc, map, st);
}

hipError_t launch_global_det(const Chunk* chunks, int64_t n_chunks, float* x, float* m,
                             float* v, float* x_rep, RepLayout rl, const GlobalScalars& sc,
                             bool broadcast, int map, hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    switch (sc.rule) {
        case kRuleLookahead:
            launch_global_det_rule<kRuleLookahead>(chunks, n_chunks, x, m, v, x_rep, rl, sc,
                                                   broadcast, map, st);
            break;
        case kRuleSignedSlowMo:
            launch_global_det_rule<kRuleSignedSlowMo>(chunks, n_chunks, x, m, v, x_rep, rl, sc,
                                                      broadcast, map, st);
            break;
        case kRuleGlobalAdamW:
            launch_global_det_rule<kRuleGlobalAdamW>(chunks, n_chunks, x, m, v, x_rep, rl, sc,
                                                     broadcast, map, st);
            break;
        default:
            launch_global_det_rule<kRuleSignMomentum>(chunks, n_chunks, x, m, v, x_rep, rl, sc,
                                                      broadcast, map, st);
            break;
    }
    return hipGetLastError();
}

hipError_t launch_global_rand(const Chunk* chunks, int64_t n_chunks, int n_tensors, float* x,
                              float* m, float* x_rep, RepLayout rl, float* u,
                              const BoundWords& bw, const GlobalScalars& sc, bool broadcast,
                              int map, hipStream_t st) {
    if (n_chunks > 0) {
        const dim3 grid = chunk_grid(n_chunks, 1), block(kBlockThreads);
        uint32_t* pm = bw.piece_max;
#define DSM_PASS1(NW) \
    hipLaunchKernelGGL(k_global_rand_pass1<NW>, grid, block, 0, st, chunks, map, x, m, x_rep, rl, u, pm, sc)
        switch (sc.n) {
            case 1: DSM_PASS1(1); break;
            case 2: DSM_PASS1(2); break;
            case 4: DSM_PASS1(4); break;
            case 8: DSM_PASS1(8); break;
            default: DSM_PASS1(0); break;
        }
#undef DSM_PASS1
    }
    if (n_tensors > 0) launch_bound_reduce(bw, n_tensors, st);
    if (n_chunks > 0)
        launch_rand_pass2(chunks, n_chunks, x, x_rep, rl, u, bw.bits, sc, broadcast, map, st);
    return hipGetLastError();
}

hipError_t launch_broadcast(const Chunk* chunks, int64_t n_chunks, const float* x, float* x_rep,
                            RepLayout rl, int n, int map, hipStream_t st) {
    if (n_chunks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_broadcast, chunk_grid(n_chunks, 1), dim3(kBlockThreads), 0, st, chunks,
                       map, x, x_rep, rl, n);
    return hipGetLastError();
}

// ---------------------------------------------------------------- static scratch

// Workspace and u staging of the contexts made by dsm_init_static, for
// callers that cannot allocate device memory.  Host code never passes this
// name to a kernel: it stands for a device address only through
// hipGetSymbolAddress, below.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

hipError_t static_scratch(void** ptr) {
    static std::mutex mu;
    static void* addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_test_stream(int kind, float* buf, int64_t n_pieces, uint32_t* words,
                              uint32_t pattern, hipStream_t st) {
    if (n_pieces == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(n_pieces)), block(kBlockThreads);
    if (kind == 0)
        hipLaunchKernelGGL(k_stream_read, grid, block, 0, st, buf, words, pattern);
    else
        hipLaunchKernelGGL(k_stream_write, grid, block, 0, st, buf, pattern);
    return hipGetLastError();
}

hipError_t launch_test_philox(uint32_t key0, uint32_t key1, uint32_t tensor, uint32_t t,
                              uint32_t q0, int64_t count, uint32_t* out, hipStream_t st) {
    if (count == 0) return hipSuccess;
    const int64_t blocks = (count + kBlockThreads - 1) / kBlockThreads;
    hipLaunchKernelGGL(k_test_philox, dim3(static_cast<unsigned>(blocks)), dim3(kBlockThreads), 0,
                       st, key0, key1, tensor, t, q0, count, out);
    return hipGetLastError();
}

}  // namespace dsm
