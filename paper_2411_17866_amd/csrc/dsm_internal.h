// Internal interface between the host runtime (dsm_runtime.cpp) and the
// gfx950 kernels (dsm_kernels.hip).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace dsm {

// Elements per work-group chunk.  A chunk never crosses a tensor boundary,
// so the per-tensor facts a kernel needs (decay flag, tensor index for the
// randomized sign's bound and Philox counter) are uniform per work-group and
// read once.  Multiple of 4 (float4) and of 256 threads x 4.
#ifndef DSM_CHUNK_ELEMS
#define DSM_CHUNK_ELEMS 16384
#endif
constexpr int kChunkElems = DSM_CHUNK_ELEMS;
static_assert(kChunkElems % 1024 == 0, "chunk must be a multiple of 256 threads x 4");
#ifndef DSM_BLOCK_THREADS
#define DSM_BLOCK_THREADS 256
#endif
constexpr int kBlockThreads = DSM_BLOCK_THREADS;
static_assert(kBlockThreads % 64 == 0 && kBlockThreads <= 1024, "whole waves, at most 1024 threads");
// float4 groups per stream in flight per thread, and loop iterations per
// work-group: a work-group takes one piece of kBlockThreads * kUnroll *
// kIters float4 groups of a chunk (build-time tuning knobs).
#ifndef DSM_UNROLL
#define DSM_UNROLL 1
#endif
#ifndef DSM_ITERS
#define DSM_ITERS 1
#endif
constexpr int kUnroll = DSM_UNROLL;
constexpr int kIters = DSM_ITERS;
constexpr int kPieceVec = kBlockThreads * kUnroll * kIters;
static_assert((kChunkElems / 4) % kPieceVec == 0, "a chunk must split into whole pieces");
// Work-groups per chunk.
constexpr int kSplit = (kChunkElems / 4) / kPieceVec;
// Arena alignment of every tensor, in elements (256 bytes).
constexpr int64_t kTensorAlign = 64;
constexpr int kMaxWorkers = 64;

// Replica buffers in 64 KiB blocks (dsm_problem.replica_layout =
// DSM_REPLICAS_BLOCKED): copy i of block b sits at element (b * n + i) *
// kRepBlockElems.  Tensors then start on a multiple of the piece size (and of
// 1024 elements), so a work-group's piece never crosses a block, and the
// arena length is a whole number of blocks.
constexpr int kRepBlockShift = 14;
constexpr int64_t kRepBlockElems = int64_t(1) << kRepBlockShift;
constexpr int64_t kPieceElems = int64_t(kPieceVec) * 4;
static_assert(kRepBlockElems % kPieceElems == 0, "a block must hold whole pieces");
constexpr int64_t kBlockedTensorAlign = kPieceElems > 1024 ? kPieceElems : 1024;

// Where copy i of a replica buffer keeps arena element e:
// (e >> shift) * block_stride + i * copy_stride + (e & (2^shift - 1)).
struct RepLayout {
    int64_t block_stride;
    int64_t copy_stride;
    int32_t shift;
    int32_t pad;
};
// n contiguous copies of d_pad elements.
inline RepLayout contiguous_copies(int64_t d_pad) { return RepLayout{0, d_pad, 62, 0}; }
// n copies interleaved in 64 KiB blocks.
inline RepLayout blocked_copies(int n) {
    return RepLayout{int64_t(n) * kRepBlockElems, kRepBlockElems, kRepBlockShift, 0};
}
// Every copy is the same single buffer (stale replicas read the global x).
inline RepLayout single_copy() { return RepLayout{0, 0, 62, 0}; }

// The replicas and their state in one allocation (dsm_problem.replica_layout =
// DSM_REPLICAS_STATE_BLOCKED): 16 KiB blocks, and block b holds the n x_rep
// copies, then the n g_rep copies, the n s1_rep copies and (AdamW) the n
// s2_rep copies of elements [4096 b, 4096 b + 4096).  Buffer j of the
// kStateBuffers starts j * n blocks into the allocation.
constexpr int kStateBlockShift = 12;
constexpr int64_t kStateBlockElems = int64_t(1) << kStateBlockShift;
static_assert(kStateBlockElems % kPieceElems == 0, "a state block must hold whole pieces");
inline RepLayout state_blocked_copies(int n, int buffers) {
    return RepLayout{int64_t(buffers) * n * kStateBlockElems, kStateBlockElems, kStateBlockShift,
                     0};
}

// Where the gradient and the base-optimizer moments of worker i keep their
// elements (the same RepLayout addressing as the replicas).
struct StateLayout {
    RepLayout g, s1, s2;
};

// One chunk of one tensor inside an arena copy.  32 bytes.
struct Chunk {
    int64_t off;      // element offset of the chunk in the arena
    int64_t j0;       // index of the chunk's first element inside its tensor
    int32_t len;      // elements in the chunk, 1..kChunkElems
    uint32_t tensor;  // tensor index p
    uint32_t decay;   // 1 if weight decay applies to the tensor
    uint32_t pad;
};
static_assert(sizeof(Chunk) == 32, "chunk descriptor is 32 bytes");

// fp32 coefficients of one AdamW local step, formed on the host in fp64 and
// rounded once.
struct AdamScalars {
    float beta1, one_minus_beta1, beta2, one_minus_beta2;
    float bc1, bc2;   // 1 - beta1^s, 1 - beta2^s
    float lr, eps, wd;
};

struct SgdScalars {
    float mu, lr;
};

// fp32 coefficients of one global step.
struct GlobalScalars {
    float beta1, beta2;
    float c1, c2;      // (1 - beta1)/gamma, (1 - beta2)/gamma
    float step;        // eta * gamma
    float lam;         // lambda (decayed tensors)
    float inv_n;       // 1/n, used only when n is a power of two (then exact)
    float n_f;         // n as float
    int32_t n;
    int32_t n_pow2;    // 1 if n is a power of two
    uint32_t key0, key1;  // Philox key (seed low, seed high)
    uint32_t t;           // outer iteration (Philox counter word 2)
    int32_t mode;         // dsm_sign
    int32_t rule;         // dsm_global_rule
    // Global AdamW (Algorithm 7) only.
    float inv_gamma;      // 1/gamma
    float one_minus_beta1, one_minus_beta2;
    float bc1, bc2;       // 1 - beta^(t+1)
    float eta, eps;
};

// How a launch's work-group index maps to its piece (the XCD map): 0, the
// index itself (XCD k takes piece k mod 8 of every chunk); 1, XCD k takes the
// k-th eighth of the grid row, in order; 2, XCD k takes whole chunks.  The
// best map of each kernel kind depends on the replica layout (measured), so
// the runtime keeps one set per layout; build-time -D settings override them.
// global: the global steps and the randomized second pass of the round end;
// copy: the broadcast of dsm_sync and the initial copy of dsm_init.
//
// A local step's map may add kInterleaveWorkers: its grid is then one row of
// pieces x workers, worker fastest, so consecutive work-groups take the same
// piece of successive workers (with the state blocked, one block at a time)
// instead of running worker by worker.
constexpr int kInterleaveWorkers = 4;
struct XcdMaps {
    int local, round_end, from_x, global, copy;
};
#ifndef DSM_MAPS_CONTIGUOUS
#define DSM_MAPS_CONTIGUOUS 1, 2, 2, 0, 0
#endif
#ifndef DSM_MAPS_BLOCKED
#define DSM_MAPS_BLOCKED 1, 2, 1, 0, 1
#endif
#ifndef DSM_MAPS_STATE_BLOCKED
#define DSM_MAPS_STATE_BLOCKED 1 + kInterleaveWorkers, 1, 1, 1, 1
#endif
constexpr XcdMaps kMapsByLayout[3] = {{DSM_MAPS_CONTIGUOUS}, {DSM_MAPS_BLOCKED},
                                      {DSM_MAPS_STATE_BLOCKED}};

// The map a local step over n_workers workers launches with: the interleaved
// order needs the whole pieces x workers row in one grid dimension, which
// holds fewer than 2^32 threads; past that the step runs worker by worker.
inline int local_map(int64_t n_chunks, int n_workers, int map) {
    const int64_t row = n_chunks * kSplit * n_workers;
    if ((map & kInterleaveWorkers) && row * kBlockThreads >= (int64_t(1) << 32))
        return map & ~kInterleaveWorkers;
    return map;
}

// Kernel launchers (dsm_kernels.hip).  All return the launch status.  The
// replica buffer x_rep is addressed through its RepLayout rl, and g_rep, s1
// and s2 through the layouts of ml; map is the launch's XCD map.
hipError_t launch_init(const Chunk* chunks, int64_t n_chunks, float* x, float* m, float* v,
                       float* x_rep, RepLayout rl, float* s1, float* s2, StateLayout ml, int n,
                       int map, hipStream_t st);
// Local steps: worker w reads its starting point from x_src through sl (its
// replica, or the shared global model with single_copy()) and writes its
// replica through rl.
hipError_t launch_local_adamw(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                              const float* x_src, RepLayout sl, const float* g_rep, float* s1,
                              float* s2, StateLayout ml, int worker0, int n_workers,
                              const AdamScalars& sc, int map, hipStream_t st);
hipError_t launch_local_sgdm(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                             const float* x_src, RepLayout sl, const float* g_rep, float* s1,
                             StateLayout ml, int worker0, int n_workers, const SgdScalars& sc,
                             int map, hipStream_t st);

// Local step of all n workers from the global model x (every replica stale):
// x is read once per element and each worker's result goes to its replica.
hipError_t launch_local_from_x(const Chunk* chunks, int64_t n_chunks, const float* x,
                               float* x_rep, RepLayout rl, const float* g_rep, float* s1,
                               float* s2, StateLayout ml, int n, bool adamw,
                               const AdamScalars& as, const SgdScalars& ss, int map,
                               hipStream_t st);

// Workspace words of the randomized sign's per-tensor bound B_p = max |u|,
// reduced in two levels without atomics.
struct BoundWords {
    uint32_t* bits;         // [n_tensors] B_p, fp32 bit patterns
    uint32_t* piece_max;    // [n_chunks * kSplit] level one: max |u| of each piece
    const int32_t* chunk0;  // [n_tensors + 1] first chunk of each tensor; last = n_chunks
};

// Arguments of the fused last-local-step + global-step launch.
struct RoundEndArgs {
    float *x, *m, *x_rep;
    RepLayout rl;           // the replicas
    const float* x_src;     // where step H starts: the replicas, or x when they are stale
    RepLayout sl;
    const float* g_rep;
    float *s1, *s2, *u;
    BoundWords bound;
    StateLayout ml;
    AdamScalars as;
    SgdScalars ss;
    GlobalScalars gs;
    int map;        // XCD map of the round-end kernel
    int map_pass2;  // and of the randomized sign's second pass
};
hipError_t launch_round_end(const Chunk* chunks, int64_t n_chunks, int n_tensors, bool adamw,
                            const RoundEndArgs& a, bool broadcast, hipStream_t st);
// Deterministic global step of any rule; v is the Global AdamW second moment.
hipError_t launch_global_det(const Chunk* chunks, int64_t n_chunks, float* x, float* m,
                             float* v, float* x_rep, RepLayout rl, const GlobalScalars& sc,
                             bool broadcast, int map, hipStream_t st);
hipError_t launch_global_rand(const Chunk* chunks, int64_t n_chunks, int n_tensors, float* x,
                              float* m, float* x_rep, RepLayout rl, float* u,
                              const BoundWords& bw, const GlobalScalars& sc, bool broadcast,
                              int map, hipStream_t st);
hipError_t launch_broadcast(const Chunk* chunks, int64_t n_chunks, const float* x, float* x_rep,
                            RepLayout rl, int n, int map, hipStream_t st);
// Streaming diagnostic over n_pieces pieces of kPieceElems floats: kind 0
// reads buf and writes 1 to words[k] for each piece k whose 32-bit patterns
// XOR to pattern; kind 1 writes the float with bit pattern `pattern`.
hipError_t launch_test_stream(int kind, float* buf, int64_t n_pieces, uint32_t* words,
                              uint32_t pattern, hipStream_t st);
hipError_t launch_test_philox(uint32_t key0, uint32_t key1, uint32_t tensor, uint32_t t,
                              uint32_t q0, int64_t count, uint32_t* out, hipStream_t st);

// The static device scratch of dsm_init_static: a file-scope array of
// kStaticScratchBytes in dsm_kernels.hip, one copy per GPU.
constexpr int64_t kStaticScratchBytes = int64_t(64) << 20;
constexpr int kMaxDevices = 64;
// Device address of the scratch on the current device, looked up once per
// device (hipGetSymbolAddress) and kept.
hipError_t static_scratch(void** ptr);

}  // namespace dsm
