// Host-only check of the library's runtime (paper_2411_17866_amd/csrc/dsm_runtime.cpp).
//
// Built with g++ and the address and undefined-behaviour sanitizers, and
// linked against stubs of the four HIP runtime calls the runtime makes and of
// the kernel launchers, so no GPU and no HIP runtime library are involved.
// "Device" buffers are host allocations and the stub copy is memcpy.  Each
// launch stub records its arguments, so the checks see exactly what every
// entry point would enqueue:
//   * dsm_layout on random valid and invalid problems;
//   * the chunk table dsm_init uploads (every element once, no chunk across a
//     tensor, decay flags);
//   * the state machine of Algorithm 1 and which source each local step reads
//     (the replica, or x after a global step without broadcast), with the
//     replica addressing of both replica layouts;
//   * the fp32 coefficients formed on the host, against long double;
//   * error paths: no device, failed launches, bad hyperparameters, NULLs;
//   * contexts driven from several threads at once (also built with the
//     thread sanitizer, where `threads` as the only argument runs just that).
// Prints "all checks passed" and exits 0, or lists the failures and exits 1.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <random>
#include <string>
#include <thread>
#include <vector>

#include "dsm.h"
#include "dsm_internal.h"

namespace {

int g_devices = 1;
int g_device = 0;            // hipGetDevice's answer
void* g_scratch = nullptr;   // host stand-in for the static device scratch
int g_scratch_lookups = 0;
hipError_t g_launch_status = hipSuccess;
std::atomic<int> g_failures{0};
std::atomic<int> g_checks{0};

#define CHECK(cond, ...)                                                          \
    do {                                                                          \
        ++g_checks;                                                               \
        if (!(cond)) {                                                            \
            ++g_failures;                                                         \
            std::fprintf(stderr, "FAIL line %d: %s: ", __LINE__, #cond);          \
            std::fprintf(stderr, __VA_ARGS__);                                    \
            std::fprintf(stderr, "\n");                                           \
        }                                                                         \
    } while (0)

struct Launch {
    std::string kind;
    const dsm::Chunk* chunks = nullptr;
    int64_t n_chunks = -1;
    int map = -1, map2 = -1;
    const float* x = nullptr;
    const float* x_rep = nullptr;
    const float* x_src = nullptr;
    dsm::RepLayout rl{-1, -1, -1, 0};  // how the launch addresses x_rep
    dsm::RepLayout sl{-1, -1, -1, 0};  // how it addresses its step's source
    const float* s2 = nullptr;
    const float* u = nullptr;
    const float* v = nullptr;
    const uint32_t* bounds = nullptr;
    const uint32_t* piece_max = nullptr;
    const int32_t* chunk0 = nullptr;
    int worker0 = -1, n_workers = -1, n_tensors = -1;
    dsm::StateLayout ml{{-1, -1, -1, 0}, {-1, -1, -1, 0}, {-1, -1, -1, 0}};
    bool broadcast = false, adamw = false;
    dsm::AdamScalars as{};
    dsm::SgdScalars ss{};
    dsm::GlobalScalars gs{};
};
std::vector<Launch> g_log;
std::mutex g_log_mu;  // launches may come from several threads (check_threads)

hipError_t record(const Launch& l) {
    std::lock_guard<std::mutex> lock(g_log_mu);
    g_log.push_back(l);
    return g_launch_status;
}

}  // namespace

// ------------------------------------------------------------ HIP runtime stubs

extern "C" {
hipError_t hipGetDeviceCount(int* count) {
    *count = g_devices;
    return hipSuccess;
}
const char* hipGetErrorString(hipError_t) { return "stubbed HIP error"; }
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind, hipStream_t) {
    std::memcpy(dst, src, bytes);
    return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipGetDevice(int* device) {
    *device = g_device;
    return hipSuccess;
}
}

// ------------------------------------------------------------ launcher stubs

namespace dsm {
hipError_t launch_init(const Chunk* chunks, int64_t n_chunks, float* x, float*, float* v,
                       float* x_rep, RepLayout rl, float*, float* s2, StateLayout ml, int n,
                       int map, hipStream_t) {
    Launch l;
    l.kind = "init";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x = x;
    l.x_rep = x_rep;
    l.rl = rl;
    l.v = v;
    l.s2 = s2;
    l.ml = ml;
    l.n_workers = n;
    return record(l);
}
hipError_t launch_local_adamw(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                              const float* x_src, RepLayout sl, const float*, float*, float* s2,
                              StateLayout ml, int worker0, int n_workers, const AdamScalars& sc,
                              int map, hipStream_t) {
    Launch l;
    l.kind = "local_adamw";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x_rep = x_rep;
    l.rl = rl;
    l.x_src = x_src;
    l.sl = sl;
    l.s2 = s2;
    l.ml = ml;
    l.worker0 = worker0;
    l.n_workers = n_workers;
    l.as = sc;
    return record(l);
}
hipError_t launch_local_sgdm(const Chunk* chunks, int64_t n_chunks, float* x_rep, RepLayout rl,
                             const float* x_src, RepLayout sl, const float*, float*,
                             StateLayout ml, int worker0, int n_workers, const SgdScalars& sc,
                             int map, hipStream_t) {
    Launch l;
    l.kind = "local_sgdm";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x_rep = x_rep;
    l.rl = rl;
    l.x_src = x_src;
    l.sl = sl;
    l.ml = ml;
    l.worker0 = worker0;
    l.n_workers = n_workers;
    l.ss = sc;
    return record(l);
}
hipError_t launch_local_from_x(const Chunk* chunks, int64_t n_chunks, const float* x,
                               float* x_rep, RepLayout rl, const float*, float*, float* s2,
                               StateLayout ml, int n, bool adamw, const AdamScalars& as,
                               const SgdScalars& ss, int map, hipStream_t) {
    Launch l;
    l.kind = "local_from_x";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x = x;
    l.x_rep = x_rep;
    l.rl = rl;
    l.s2 = s2;
    l.ml = ml;
    l.n_workers = n;
    l.adamw = adamw;
    l.as = as;
    l.ss = ss;
    return record(l);
}
hipError_t launch_round_end(const Chunk* chunks, int64_t n_chunks, int n_tensors, bool adamw,
                            const RoundEndArgs& a, bool broadcast, hipStream_t) {
    Launch l;
    l.kind = "round_end";
    l.map = a.map;
    l.map2 = a.map_pass2;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.n_tensors = n_tensors;
    l.adamw = adamw;
    l.x = a.x;
    l.x_rep = a.x_rep;
    l.rl = a.rl;
    l.x_src = a.x_src;
    l.sl = a.sl;
    l.s2 = a.s2;
    l.u = a.u;
    l.bounds = a.bound.bits;
    l.piece_max = a.bound.piece_max;
    l.chunk0 = a.bound.chunk0;
    l.ml = a.ml;
    l.broadcast = broadcast;
    l.as = a.as;
    l.ss = a.ss;
    l.gs = a.gs;
    return record(l);
}
hipError_t launch_global_det(const Chunk* chunks, int64_t n_chunks, float* x, float*, float* v,
                             float* x_rep, RepLayout rl, const GlobalScalars& sc, bool broadcast,
                             int map, hipStream_t) {
    Launch l;
    l.kind = "global_det";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x = x;
    l.v = v;
    l.x_rep = x_rep;
    l.rl = rl;
    l.gs = sc;
    l.broadcast = broadcast;
    return record(l);
}
hipError_t launch_global_rand(const Chunk* chunks, int64_t n_chunks, int n_tensors, float* x,
                              float*, float* x_rep, RepLayout rl, float* u, const BoundWords& bw,
                              const GlobalScalars& sc, bool broadcast, int map, hipStream_t) {
    Launch l;
    l.kind = "global_rand";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.n_tensors = n_tensors;
    l.x = x;
    l.x_rep = x_rep;
    l.rl = rl;
    l.u = u;
    l.bounds = bw.bits;
    l.piece_max = bw.piece_max;
    l.chunk0 = bw.chunk0;
    l.gs = sc;
    l.broadcast = broadcast;
    return record(l);
}
hipError_t launch_broadcast(const Chunk* chunks, int64_t n_chunks, const float* x, float* x_rep,
                            RepLayout rl, int n, int map, hipStream_t) {
    Launch l;
    l.kind = "broadcast";
    l.map = map;
    l.chunks = chunks;
    l.n_chunks = n_chunks;
    l.x = x;
    l.x_rep = x_rep;
    l.rl = rl;
    l.n_workers = n;
    return record(l);
}
hipError_t static_scratch(void** ptr) {
    ++g_scratch_lookups;
    if (g_scratch == nullptr) {
        g_scratch = std::aligned_alloc(256, static_cast<size_t>(kStaticScratchBytes));
        std::memset(g_scratch, 0x5A, static_cast<size_t>(kStaticScratchBytes));
    }
    *ptr = g_scratch;
    return hipSuccess;
}
hipError_t launch_test_stream(int kind, float* buf, int64_t n_pieces, uint32_t* words,
                              uint32_t, hipStream_t) {
    Launch l;
    l.kind = kind == 0 ? "stream_read" : "stream_write";
    l.x = buf;
    l.n_chunks = n_pieces;
    l.bounds = words;
    return record(l);
}
hipError_t launch_test_philox(uint32_t, uint32_t, uint32_t, uint32_t, uint32_t, int64_t,
                              uint32_t* out, hipStream_t) {
    Launch l;
    l.kind = "test_philox";
    l.bounds = out;
    return record(l);
}
}  // namespace dsm

// ------------------------------------------------------------ helpers

namespace {

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

bool same_layout(const dsm::RepLayout& a, const dsm::RepLayout& b) {
    return a.block_stride == b.block_stride && a.copy_stride == b.copy_stride && a.shift == b.shift;
}

// The replica layout a launch must use, written out from dsm.h: contiguous
// copies at i * d_pad, 64 KiB blocks at ((e / 16384) * n + i) * 16384, or
// state blocks at ((e / 4096) * B * n + i) * 4096 from each buffer's start.
dsm::RepLayout expected_layout(int replica_layout, int n, int64_t arena, int buffers) {
    if (replica_layout == DSM_REPLICAS_BLOCKED) return dsm::RepLayout{int64_t(n) * 16384, 16384, 14, 0};
    if (replica_layout == DSM_REPLICAS_STATE_BLOCKED)
        return dsm::RepLayout{int64_t(buffers) * n * 4096, 4096, 12, 0};
    return dsm::RepLayout{0, arena, 62, 0};
}

bool same_state(const dsm::StateLayout& a, const dsm::RepLayout& g) {
    return same_layout(a.g, g) && same_layout(a.s1, g) && same_layout(a.s2, g);
}

// The element index a RepLayout gives copy i of element e.
int64_t rep_element(const dsm::RepLayout& L, int64_t i, int64_t e) {
    const int64_t mask = (int64_t(1) << L.shift) - 1;
    return (e >> L.shift) * L.block_stride + i * L.copy_stride + (e & mask);
}

int64_t tensor_align(int replica_layout) {
    return replica_layout != DSM_REPLICAS_CONTIGUOUS ? std::max<int64_t>(1024, dsm::kPieceElems) : 64;
}

int64_t arena_block(int replica_layout) {
    return replica_layout == DSM_REPLICAS_BLOCKED ? 16384
           : replica_layout == DSM_REPLICAS_STATE_BLOCKED ? 4096 : 1;
}

struct Problem {
    std::vector<int64_t> numel;
    std::vector<uint8_t> decay;
    dsm_problem p{};
    Problem(std::vector<int64_t> ne, int n, int H, int base, std::vector<uint8_t> dec = {},
            int layout = DSM_REPLICAS_CONTIGUOUS)
        : numel(std::move(ne)), decay(std::move(dec)) {
        p.n_workers = n;
        p.local_steps = H;
        p.n_tensors = static_cast<int32_t>(numel.size());
        p.base = base;
        p.numel = numel.empty() ? nullptr : numel.data();
        p.decay = decay.empty() ? nullptr : decay.data();
        p.replica_layout = layout;
    }
};

// Host allocations standing in for the caller's device buffers.
struct Buffers {
    std::vector<void*> owned;
    dsm_buffers b{};
    int64_t arena = 0;
    dsm::RepLayout rep{};  // the replica layout every launch must pass
    dsm::RepLayout state{};  // and the layout of g_rep, s1_rep and s2_rep
    dsm::XcdMaps maps{};     // the XCD maps of the problem's layout
    float* alloc(int64_t floats) {
        const size_t bytes = static_cast<size_t>(round_up(std::max<int64_t>(floats, 1) * 4, 256));
        void* p = std::aligned_alloc(256, bytes);
        std::memset(p, 0, bytes);
        owned.push_back(p);
        return static_cast<float*>(p);
    }
    Buffers(const Problem& P, bool randomized, bool global_adamw) {
        int64_t ws = 0;
        std::vector<int64_t> off(P.numel.size() + 1);
        dsm_status st = dsm_layout(&P.p, &arena, off.data(), &ws);
        CHECK(st == DSM_OK, "layout of a valid problem");
        const int n = P.p.n_workers;
        const bool adamw = P.p.base == DSM_BASE_ADAMW;
        const int nb = adamw ? 4 : 3;
        rep = expected_layout(P.p.replica_layout, n, arena, nb);
        if (P.p.replica_layout >= 0 && P.p.replica_layout <= 2)
            maps = dsm::kMapsByLayout[P.p.replica_layout];
        b.x = alloc(arena);
        b.m = alloc(arena);
        if (P.p.replica_layout == DSM_REPLICAS_STATE_BLOCKED) {
            // One allocation; each buffer starts j * n blocks in.
            state = rep;
            b.x_rep = alloc(nb * n * arena);
            b.g_rep = b.x_rep + n * 4096;
            b.s1_rep = b.x_rep + 2 * n * 4096;
            b.s2_rep = adamw ? b.x_rep + 3 * n * 4096 : nullptr;
        } else {
            state = dsm::RepLayout{0, arena, 62, 0};
            b.x_rep = alloc(n * arena);
            b.g_rep = alloc(n * arena);
            b.s1_rep = alloc(n * arena);
            b.s2_rep = adamw ? alloc(n * arena) : nullptr;
        }
        b.u_scratch = randomized ? alloc(arena) : nullptr;
        b.v = global_adamw ? alloc(arena) : nullptr;
        b.workspace = alloc(ws / 4 + 64);
        // Garbage, so that a part the runtime fails to upload shows.
        std::memset(b.workspace, 0xA5, static_cast<size_t>(ws));
        b.workspace_bytes = ws;
        b.stream = nullptr;
    }
    ~Buffers() {
        for (void* p : owned) std::free(p);
    }
    Buffers(const Buffers&) = delete;
    Buffers& operator=(const Buffers&) = delete;
};

dsm_local_hparams adam_hp() { return dsm_local_hparams{1e-3f, 0.9f, 0.95f, 1e-8f, 0.1f}; }
dsm_local_hparams sgd_hp() { return dsm_local_hparams{0.05f, 0.5f, 0.0f, 0.0f, 0.0f}; }
dsm_global_hparams glob_hp(int mode = DSM_SIGN_DET, int rule = DSM_RULE_SIGN_MOMENTUM) {
    dsm_global_hparams h{};
    h.gamma = 1e-3f;
    h.eta = 0.8f;
    h.beta1 = 0.95f;
    h.beta2 = 0.98f;
    h.lambda = 0.1f;
    h.mode = mode;
    h.seed = 0x0123456789ABCDEFull;
    h.rule = rule;
    h.eps = 1e-8f;
    return h;
}

// fp32 rounding of a long double value, as the host coefficients promise
// (fp64 formation rounded once can sit one fp32 ulp away at a tie boundary).
bool close_f32(float got, long double want) {
    const float w = static_cast<float>(want);
    return got == w || got == std::nextafter(w, INFINITY) || got == std::nextafter(w, -INFINITY);
}

// ------------------------------------------------------------ checks

void check_layout_fuzz() {
    std::mt19937_64 rng(12345);
    const int64_t special[] = {0, 1, 3, 63, 64, 65, 1000, 16383, 16384, 16385, 40003, 100000};
    for (int iter = 0; iter < 3000; ++iter) {
        const int nt = static_cast<int>(rng() % 40);
        std::vector<int64_t> ne(nt);
        for (auto& v : ne)
            v = (rng() % 3) ? special[rng() % 12] : static_cast<int64_t>(rng() % 300000);
        int n = 1 + static_cast<int>(rng() % 64), H = 1 + static_cast<int>(rng() % 30);
        int base = static_cast<int>(rng() % 2);
        int layout = static_cast<int>(rng() % 3);
        std::vector<uint8_t> dec;
        if (rng() % 2) {
            dec.resize(nt);
            for (auto& d : dec) d = static_cast<uint8_t>(rng() % 2);
        }
        // One in four problems gets exactly one invalid field.
        const int bad = (rng() % 4 == 0) ? 1 + static_cast<int>(rng() % 7) : 0;
        if (bad == 1) n = (rng() % 2) ? 0 : 65;
        if (bad == 2) H = 0;
        if (bad == 3) base = 2 + static_cast<int>(rng() % 5);
        if (bad == 4 && nt > 0) ne[rng() % nt] = -1 - static_cast<int64_t>(rng() % 5);
        if (bad == 5 && nt > 0) ne[rng() % nt] = (int64_t(1) << 34) + static_cast<int64_t>(rng() % 7);
        if (bad == 6) layout = (rng() % 2) ? -1 : 3 + static_cast<int>(rng() % 5);
        const bool invalid =
            bad == 1 || bad == 2 || bad == 3 || bad == 6 || ((bad == 4 || bad == 5) && nt > 0);
        Problem P(ne, n, H, base, dec, layout);
        int64_t arena = -7, ws = -7;
        std::vector<int64_t> off(nt + 1, -7);
        const dsm_status st = dsm_layout(&P.p, &arena, off.data(), &ws);
        if (invalid) {
            CHECK(st == DSM_ERR_INVALID_ARG, "iter %d: invalid field %d accepted (status %d)", iter,
                  bad, st);
            CHECK(std::strlen(dsm_last_error(nullptr)) > 0, "iter %d: no error text", iter);
            CHECK(arena == -7 && ws == -7, "iter %d: outputs written on error", iter);
            continue;
        }
        CHECK(st == DSM_OK, "iter %d: valid problem rejected: %s", iter, dsm_last_error(nullptr));
        int64_t o = 0, chunks = 0;
        for (int i = 0; i < nt; ++i) {
            CHECK(off[i] == o, "iter %d: offset %d is %lld, expected %lld", iter, i,
                  static_cast<long long>(off[i]), static_cast<long long>(o));
            o += round_up(ne[i], tensor_align(layout));
            chunks += (ne[i] + dsm::kChunkElems - 1) / dsm::kChunkElems;
        }
        o = round_up(o, arena_block(layout));
        CHECK(arena == o, "iter %d: arena %lld, expected %lld", iter, static_cast<long long>(arena),
              static_cast<long long>(o));
        CHECK(ws == round_up(chunks * 32, 256) + round_up(int64_t(nt) * 4, 256) +
                        (nt > 0 ? round_up((int64_t(nt) + 1) * 4, 256) : 0) +
                        round_up(chunks * dsm::kSplit * 4, 256),
              "iter %d: workspace %lld", iter, static_cast<long long>(ws));
        CHECK(off[nt] == -7, "iter %d: wrote past tensor_offsets", iter);
    }
    // NULL outputs are allowed; a NULL problem is an argument error.
    Problem P({5, 7}, 2, 2, DSM_BASE_ADAMW);
    CHECK(dsm_layout(&P.p, nullptr, nullptr, nullptr) == DSM_OK, "NULL outputs");
    CHECK(dsm_layout(nullptr, nullptr, nullptr, nullptr) == DSM_ERR_INVALID_ARG, "NULL problem");
    Problem Q({5, 7}, 2, 2, DSM_BASE_ADAMW);
    Q.p.numel = nullptr;
    CHECK(dsm_layout(&Q.p, nullptr, nullptr, nullptr) == DSM_ERR_INVALID_ARG, "NULL numel");
}

// The uploaded chunk table covers every element of every tensor once, in
// order, with no chunk crossing a tensor, and carries the decay flags.
void check_chunk_table(const Problem& P, const Buffers& B, const Launch& init) {
    const auto* c = static_cast<const dsm::Chunk*>(B.b.workspace);
    CHECK(init.chunks == c, "init reads the chunk table from the workspace");
    int64_t k = 0, off = 0;
    for (size_t i = 0; i < P.numel.size(); ++i) {
        const uint32_t dec = P.decay.empty() ? 1u : (P.decay[i] ? 1u : 0u);
        for (int64_t j = 0; j < P.numel[i]; ++k) {
            CHECK(k < init.n_chunks, "tensor %zu element %lld beyond the chunk table", i,
                  static_cast<long long>(j));
            if (k >= init.n_chunks) return;
            CHECK(c[k].tensor == i && c[k].j0 == j && c[k].off == off + j,
                  "chunk %lld: tensor %u j0 %lld off %lld", static_cast<long long>(k), c[k].tensor,
                  static_cast<long long>(c[k].j0), static_cast<long long>(c[k].off));
            CHECK(c[k].len >= 1 && c[k].len <= dsm::kChunkElems && j + c[k].len <= P.numel[i],
                  "chunk %lld length %d", static_cast<long long>(k), c[k].len);
            CHECK(c[k].decay == dec, "chunk %lld decay flag", static_cast<long long>(k));
            j += c[k].len;
        }
        off += round_up(P.numel[i], tensor_align(P.p.replica_layout));
    }
    CHECK(k == init.n_chunks, "chunk count %lld, table has %lld", static_cast<long long>(k),
          static_cast<long long>(init.n_chunks));
}

// The randomized sign's bound words in the workspace, each part at a
// 256-byte boundary: the bounds after the chunk table, then the first chunk
// of each tensor (uploaded at init, n_tensors + 1 words), then one
// piece-maximum word per work-group piece.
void check_bound_words(const Problem& P, const Buffers& B, const uint32_t* bits,
                       const int32_t* chunk0, const uint32_t* piece_max, const char* what) {
    const auto* ws = static_cast<const char*>(B.b.workspace);
    const int64_t nt = static_cast<int64_t>(P.numel.size());
    std::vector<int32_t> want;
    int64_t n_chunks = 0;
    for (int64_t ne : P.numel) {
        want.push_back(static_cast<int32_t>(n_chunks));
        n_chunks += (ne + dsm::kChunkElems - 1) / dsm::kChunkElems;
    }
    want.push_back(static_cast<int32_t>(n_chunks));
    const int64_t bounds_off = round_up(n_chunks * 32, 256);
    const int64_t chunk0_off = bounds_off + round_up(nt * 4, 256);
    const int64_t pmax_off = chunk0_off + round_up((nt + 1) * 4, 256);
    CHECK(reinterpret_cast<const char*>(bits) == ws + bounds_off,
          "%s: bound words follow the chunk table", what);
    CHECK(reinterpret_cast<const char*>(chunk0) == ws + chunk0_off,
          "%s: tensor chunk index follows the bounds", what);
    CHECK(reinterpret_cast<const char*>(piece_max) == ws + pmax_off,
          "%s: piece maxima follow the tensor chunk index", what);
    CHECK(pmax_off + n_chunks * dsm::kSplit * 4 <= B.b.workspace_bytes,
          "%s: piece maxima inside the workspace", what);
    CHECK(std::memcmp(ws + chunk0_off, want.data(), want.size() * sizeof(int32_t)) == 0,
          "%s: uploaded tensor chunk index", what);
}

void check_init_and_chunks() {
    const std::vector<std::vector<int64_t>> shapes = {
        {1, 3, 4, 5, 63, 64, 65, 0, 1000, 16383, 16384, 16385, 40003}, {0}, {16384 * 3}, {7}};
    for (size_t s = 0; s < shapes.size(); ++s) {
        std::vector<uint8_t> dec(shapes[s].size());
        for (size_t i = 0; i < dec.size(); ++i) dec[i] = (i % 3 != 1);
        for (int with_decay = 0; with_decay < 6; ++with_decay) {
            const int layout = with_decay / 2;   // contiguous, blocked, state-blocked
            Problem P(shapes[s], 3, 2, DSM_BASE_ADAMW,
                      with_decay % 2 ? dec : std::vector<uint8_t>{}, layout);
            Buffers B(P, false, true);
            g_log.clear();
            dsm_ctx* ctx = nullptr;
            CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init: %s", dsm_last_error(nullptr));
            const bool empty = B.arena == 0;
            CHECK(g_log.size() == (empty ? 0u : 1u), "init launches %zu kernels", g_log.size());
            if (!empty && !g_log.empty()) {
                const Launch& l = g_log[0];
                CHECK(l.kind == "init" && l.x == B.b.x && l.x_rep == B.b.x_rep && l.v == B.b.v &&
                          l.s2 == B.b.s2_rep && same_state(l.ml, B.state) && l.n_workers == 3 &&
                          same_layout(l.rl, B.rep) && l.map == B.maps.copy,
                      "init arguments");
                check_chunk_table(P, B, l);
            }
            if (!P.numel.empty()) {
                int64_t n_chunks = 0;
                for (int64_t ne : P.numel) n_chunks += (ne + dsm::kChunkElems - 1) / dsm::kChunkElems;
                const char* ws = static_cast<const char*>(B.b.workspace);
                const int64_t bo = round_up(n_chunks * 32, 256);
                const int64_t co = bo + round_up(static_cast<int64_t>(P.numel.size()) * 4, 256);
                const int64_t po = co + round_up((static_cast<int64_t>(P.numel.size()) + 1) * 4, 256);
                check_bound_words(P, B, reinterpret_cast<const uint32_t*>(ws + bo),
                                  reinterpret_cast<const int32_t*>(ws + co),
                                  reinterpret_cast<const uint32_t*>(ws + po), "init");
            }
            CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
        }
    }
}

void check_init_rejections() {
    Problem P({1000, 7}, 2, 3, DSM_BASE_ADAMW);
    {
        Buffers B(P, false, false);
        dsm_ctx* ctx = reinterpret_cast<dsm_ctx*>(0x1);
        B.b.s2_rep = nullptr;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_INVALID_ARG && ctx == nullptr,
              "AdamW without s2_rep");
    }
    {
        Buffers B(P, false, false);
        dsm_ctx* ctx = nullptr;
        B.b.m = reinterpret_cast<float*>(reinterpret_cast<char*>(B.b.m) + 4);
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_INVALID_ARG, "misaligned m");
    }
    {
        Buffers B(P, false, false);
        dsm_ctx* ctx = nullptr;
        B.b.workspace_bytes -= 1;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_INVALID_ARG, "short workspace");
        CHECK(std::strstr(dsm_last_error(nullptr), "workspace") != nullptr, "workspace message");
    }
    {
        Buffers B(P, false, false);
        dsm_ctx* ctx = nullptr;
        CHECK(dsm_init(&P.p, &B.b, nullptr) == DSM_ERR_INVALID_ARG, "NULL out");
        CHECK(dsm_init(&P.p, nullptr, &ctx) == DSM_ERR_INVALID_ARG, "NULL buffers");
        g_devices = 0;
        g_log.clear();
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_HIP && ctx == nullptr, "no device");
        CHECK(std::strstr(dsm_last_error(nullptr), "no HIP device") != nullptr, "device message");
        CHECK(g_log.empty(), "no launch without a device");
        g_devices = 1;
        g_launch_status = hipErrorLaunchFailure;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_HIP && ctx == nullptr, "failed init launch");
        g_launch_status = hipSuccess;
    }
}

// Which replica source each local launch reads, for workers [w0, w0 + nw).
void expect_local(const Launch& l, const Buffers& B, bool adamw, bool from_x, int w0, int nw,
                  const char* what) {
    CHECK(l.kind == (adamw ? "local_adamw" : "local_sgdm"), "%s: kind %s", what, l.kind.c_str());
    CHECK(l.x_rep == B.b.x_rep && same_state(l.ml, B.state) && same_layout(l.rl, B.rep) &&
              l.map == B.maps.local,
          "%s: replica buffer", what);
    CHECK(l.x_src == (from_x ? B.b.x : B.b.x_rep) &&
              same_layout(l.sl, from_x ? dsm::RepLayout{0, 0, 62, 0} : B.rep),
          "%s: source %s expected", what, from_x ? "x" : "x_rep");
    CHECK(l.worker0 == w0 && l.n_workers == nw, "%s: workers [%d, +%d) expected, got [%d, +%d)",
          what, w0, nw, l.worker0, l.n_workers);
    CHECK(l.chunks == B.b.workspace, "%s: chunk table", what);
}

void check_state_machine_adamw(int layout) {
    Problem P({100, 16385, 7}, 5, 3, DSM_BASE_ADAMW, {1, 1, 0}, layout);
    Buffers B(P, true, false);
    dsm_ctx* ctx = nullptr;
    CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init");
    const dsm_local_hparams lh = adam_hp();
    const dsm_global_hparams gh = glob_hp();
    g_log.clear();
    // Round t = 0: all workers, then worker 2 alone: a global step is refused
    // until every worker has taken H steps; a step past H is refused.
    CHECK(dsm_local_step(ctx, -1, 1, &lh) == DSM_OK, "local all");
    CHECK(dsm_local_step(ctx, 2, 2, &lh) == DSM_OK, "local worker 2");
    CHECK(dsm_global_step(ctx, 0, &gh, 1) == DSM_ERR_STATE, "global before H");
    CHECK(dsm_round_end(ctx, 3, &lh, 0, &gh, 1) == DSM_ERR_STATE, "round end with uneven counts");
    CHECK(dsm_local_step(ctx, 2, 3, &lh) == DSM_OK, "worker 2 step 3");
    CHECK(dsm_local_step(ctx, 2, 4, &lh) == DSM_ERR_STATE, "worker 2 past H");
    CHECK(dsm_local_step(ctx, -1, 4, &lh) == DSM_ERR_STATE, "all workers past H for worker 2");
    CHECK(g_log.size() == 3, "three launches so far, got %zu", g_log.size());
    if (g_log.size() == 3) {
        expect_local(g_log[0], B, true, false, 0, 5, "round 0 all");
        expect_local(g_log[1], B, true, false, 2, 1, "round 0 worker 2");
        expect_local(g_log[2], B, true, false, 2, 1, "round 0 worker 2 again");
    }
    for (int w : {0, 1, 3, 4}) CHECK(dsm_local_step(ctx, w, 2, &lh) == DSM_OK, "worker %d", w);
    for (int w : {0, 1, 3, 4}) CHECK(dsm_local_step(ctx, w, 3, &lh) == DSM_OK, "worker %d", w);
    CHECK(dsm_read_bounds(ctx, nullptr, 0) == DSM_ERR_STATE, "bounds before a randomized step");
    // Global step without broadcast: every replica becomes stale.
    g_log.clear();
    CHECK(dsm_global_step(ctx, 0, &gh, 0) == DSM_OK, "global, no broadcast");
    CHECK(g_log.size() == 1 && g_log[0].kind == "global_det" && !g_log[0].broadcast &&
              g_log[0].x == B.b.x && g_log[0].x_rep == B.b.x_rep && same_layout(g_log[0].rl, B.rep) &&
              g_log[0].map == B.maps.global,
          "global launch");
    // Round t = 1: worker 1 first (reads x), then all: runs [0], [1], [2, 5) with
    // sources x, x_rep, x.
    g_log.clear();
    CHECK(dsm_local_step(ctx, 1, 4, &lh) == DSM_OK, "stale worker 1");
    CHECK(dsm_local_step(ctx, -1, 5, &lh) == DSM_OK, "mixed all");
    CHECK(g_log.size() == 4, "four launches, got %zu", g_log.size());
    if (g_log.size() == 4) {
        expect_local(g_log[0], B, true, true, 1, 1, "stale worker 1");
        expect_local(g_log[1], B, true, true, 0, 1, "run [0]");
        expect_local(g_log[2], B, true, false, 1, 1, "run [1]");
        expect_local(g_log[3], B, true, true, 2, 3, "run [2, 5)");
    }
    // Workers 0 and 2-4 have 1 step, worker 1 has 2: finish to H - 1 = 2
    // and end the round fused, randomized, with broadcast.
    for (int w : {0, 2, 3, 4}) CHECK(dsm_local_step(ctx, w, 6, &lh) == DSM_OK, "worker %d", w);
    const dsm_global_hparams gr = glob_hp(DSM_SIGN_RAND_FLIP);
    g_log.clear();
    CHECK(dsm_round_end(ctx, 7, &lh, 1, &gr, 1) == DSM_OK, "fused round end: %s",
          dsm_last_error(ctx));
    CHECK(g_log.size() == 1, "one round-end launch");
    if (g_log.size() == 1) {
        const Launch& l = g_log[0];
        CHECK(l.kind == "round_end" && l.adamw && l.broadcast && l.n_tensors == 3, "round end");
        CHECK(l.x_src == B.b.x_rep && same_layout(l.sl, B.rep) && same_layout(l.rl, B.rep),
              "round end reads the replicas");
        CHECK(l.map == B.maps.round_end && l.map2 == B.maps.global, "round end XCD maps");
        CHECK(l.u == B.b.u_scratch && l.s2 == B.b.s2_rep, "round end buffers");
        check_bound_words(P, B, l.bounds, l.chunk0, l.piece_max, "round end");
        CHECK(l.gs.mode == DSM_SIGN_RAND_FLIP && l.gs.t == 1 && l.gs.key0 == 0x89ABCDEFu &&
                  l.gs.key1 == 0x01234567u,
              "Philox key and counter word");
    }
    // The bounds of that step are read back from the workspace.
    if (!g_log.empty()) {
        auto* words = const_cast<uint32_t*>(g_log[0].bounds);
        const float want[3] = {0.5f, 2.0f, 0.0f};
        std::memcpy(words, want, sizeof want);
        float got[3] = {-1, -1, -1};
        float small[2] = {-1, -1};
        CHECK(dsm_read_bounds(ctx, small, 2) == DSM_ERR_INVALID_ARG, "capacity below n_tensors");
        CHECK(small[0] == -1 && small[1] == -1, "nothing written on a short array");
        CHECK(dsm_read_bounds(ctx, got, 3) == DSM_OK, "read bounds");
        CHECK(std::memcmp(got, want, sizeof want) == 0, "bounds round trip");
        CHECK(dsm_read_bounds(ctx, nullptr, 3) == DSM_ERR_INVALID_ARG, "NULL bounds output");
    }
    // Variants are refused by the fused round end; round end with H - 1
    // steps only.
    dsm_global_hparams gl = glob_hp(DSM_SIGN_DET, DSM_RULE_LOOKAHEAD);
    CHECK(dsm_local_step(ctx, -1, 8, &lh) == DSM_OK, "round t = 2, step 1");
    CHECK(dsm_local_step(ctx, -1, 9, &lh) == DSM_OK, "round t = 2, step 2");
    CHECK(dsm_round_end(ctx, 10, &lh, 2, &gl, 1) == DSM_ERR_UNSUPPORTED, "variant in round end");
    gl.mode = DSM_SIGN_RAND_FLIP;
    CHECK(dsm_round_end(ctx, 10, &lh, 2, &gl, 1) == DSM_ERR_INVALID_ARG, "randomized variant");
    // dsm_sync resets the round: local counts restart at 0.
    g_log.clear();
    CHECK(dsm_sync(ctx) == DSM_OK, "sync");
    CHECK(g_log.size() == 1 && g_log[0].kind == "broadcast" && g_log[0].n_workers == 5 &&
              g_log[0].x == B.b.x && g_log[0].x_rep == B.b.x_rep && same_layout(g_log[0].rl, B.rep) &&
              g_log[0].map == B.maps.copy,
          "broadcast launch");
    for (int k = 0; k < 3; ++k) CHECK(dsm_local_step(ctx, -1, 11 + k, &lh) == DSM_OK, "after sync");
    CHECK(dsm_local_step(ctx, -1, 14, &lh) == DSM_ERR_STATE, "H after sync");
    // A failed launch reports DSM_ERR_HIP and leaves the round where it was.
    g_launch_status = hipErrorLaunchFailure;
    CHECK(dsm_global_step(ctx, 3, &gh, 1) == DSM_ERR_HIP, "failed global launch");
    g_launch_status = hipSuccess;
    CHECK(dsm_global_step(ctx, 3, &gh, 1) == DSM_OK, "global after the failure");
    CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
}

void check_state_machine_sgd_h1(int layout) {
    // H = 1: the fused round end takes the only local step; after a lazy
    // round end it reads x, after a broadcast the replicas.
    Problem P({64, 65}, 3, 1, DSM_BASE_SGD_MOMENTUM, {}, layout);
    Buffers B(P, false, false);
    dsm_ctx* ctx = nullptr;
    CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init");
    const dsm_local_hparams lh = sgd_hp();
    const dsm_global_hparams gh = glob_hp();
    g_log.clear();
    CHECK(dsm_round_end(ctx, 1, &lh, 0, &gh, 0) == DSM_OK, "round end 0 (lazy)");
    CHECK(dsm_round_end(ctx, 2, &lh, 1, &gh, 1) == DSM_OK, "round end 1 (broadcast)");
    CHECK(dsm_round_end(ctx, 3, &lh, 2, &gh, 1) == DSM_OK, "round end 2");
    CHECK(g_log.size() == 3, "three launches");
    if (g_log.size() == 3) {
        const dsm::RepLayout x_only{0, 0, 62, 0};
        CHECK(g_log[0].x_src == B.b.x_rep && same_layout(g_log[0].sl, B.rep), "fresh after init");
        CHECK(g_log[1].x_src == B.b.x && same_layout(g_log[1].sl, x_only),
              "stale after lazy round end");
        CHECK(g_log[2].x_src == B.b.x_rep && same_layout(g_log[2].sl, B.rep),
              "fresh after broadcast");
        for (const Launch& l : g_log) CHECK(same_layout(l.rl, B.rep), "round end replica layout");
        CHECK(!g_log[0].adamw && g_log[0].ss.mu == 0.5f && g_log[0].ss.lr == 0.05f, "SGD scalars");
        CHECK(g_log[0].s2 == nullptr, "no second moment for SGD");
    }
    CHECK(dsm_local_step(ctx, -1, 4, &lh) == DSM_OK, "split step");
    CHECK(dsm_round_end(ctx, 5, &lh, 3, &gh, 1) == DSM_ERR_STATE, "round end after the H-th step");
    const dsm_global_hparams gr = glob_hp(DSM_SIGN_RAND_ZERO);
    CHECK(dsm_global_step(ctx, 3, &gr, 1) == DSM_ERR_INVALID_ARG, "randomized without u_scratch");
    dsm_global_hparams ga = glob_hp(DSM_SIGN_DET, DSM_RULE_GLOBAL_ADAMW);
    CHECK(dsm_global_step(ctx, 3, &ga, 1) == DSM_ERR_INVALID_ARG, "Global AdamW without v");
    CHECK(dsm_global_step(ctx, 3, &gh, 1) == DSM_OK, "global");
    CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
}

// After a global step without broadcast every replica is stale: a local
// step of all workers reads x once in one launch (n >= 2); one worker, or
// n = 1, keeps the per-worker launch reading x.
void check_local_from_x(int layout) {
    for (int base : {DSM_BASE_ADAMW, DSM_BASE_SGD_MOMENTUM}) {
        const bool adamw = base == DSM_BASE_ADAMW;
        const dsm_local_hparams lh = adamw ? adam_hp() : sgd_hp();
        const dsm_global_hparams gh = glob_hp();
        for (int n : {1, 2, 3, 8}) {
            Problem P({100, 16385}, n, 2, base, {}, layout);
            Buffers B(P, false, false);
            dsm_ctx* ctx = nullptr;
            CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init");
            for (int k = 0; k < 2; ++k) CHECK(dsm_local_step(ctx, -1, k + 1, &lh) == DSM_OK, "local");
            CHECK(dsm_global_step(ctx, 0, &gh, 0) == DSM_OK, "lazy global step");
            g_log.clear();
            CHECK(dsm_local_step(ctx, -1, 3, &lh) == DSM_OK, "first local step after it");
            CHECK(g_log.size() == 1, "one launch, got %zu", g_log.size());
            if (g_log.size() == 1) {
                const Launch& l = g_log[0];
                if (n >= 2) {
                    CHECK(l.kind == "local_from_x" && l.x == B.b.x && l.x_rep == B.b.x_rep &&
                              same_state(l.ml, B.state) && l.n_workers == n && l.adamw == adamw &&
                              l.s2 == B.b.s2_rep && l.chunks == B.b.workspace &&
                              same_layout(l.rl, B.rep) && l.map == B.maps.from_x,
                          "n = %d: all-worker launch from x", n);
                } else {
                    expect_local(l, B, adamw, true, 0, 1, "n = 1 from x");
                }
            }
            // The step counts and clears the stale flags like any local step.
            CHECK(dsm_local_step(ctx, -1, 4, &lh) == DSM_OK, "second local step");
            if (g_log.size() == 2) expect_local(g_log[1], B, adamw, false, 0, n, "then from replicas");
            CHECK(dsm_local_step(ctx, -1, 5, &lh) == DSM_ERR_STATE, "H reached");
            CHECK(dsm_global_step(ctx, 1, &gh, 0) == DSM_OK, "lazy again");
            // One worker alone after a lazy step still uses the per-worker path.
            g_log.clear();
            CHECK(dsm_local_step(ctx, 0, 5, &lh) == DSM_OK, "worker 0 alone");
            if (g_log.size() == 1) expect_local(g_log[0], B, adamw, true, 0, 1, "worker 0 from x");
            CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
        }
    }
}

void check_coefficients() {
    Problem P({300}, 3, 1000000, DSM_BASE_ADAMW);
    Buffers B(P, false, true);
    dsm_ctx* ctx = nullptr;
    CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init");
    const dsm_local_hparams lh = adam_hp();
    const int64_t steps[] = {1, 2, 3, 10, 100, 1000, 54321, 999999};
    for (int64_t s : steps) {
        g_log.clear();
        CHECK(dsm_local_step(ctx, -1, s, &lh) == DSM_OK, "local step %lld", static_cast<long long>(s));
        if (g_log.size() != 1) continue;
        const dsm::AdamScalars& a = g_log[0].as;
        const long double b1 = lh.beta1, b2 = lh.beta2;
        CHECK(close_f32(a.bc1, 1.0L - std::pow(b1, static_cast<long double>(s))), "bc1 at s=%lld: %.9g",
              static_cast<long long>(s), a.bc1);
        CHECK(close_f32(a.bc2, 1.0L - std::pow(b2, static_cast<long double>(s))), "bc2 at s=%lld: %.9g",
              static_cast<long long>(s), a.bc2);
        CHECK(a.one_minus_beta1 == static_cast<float>(1.0L - b1) &&
                  a.one_minus_beta2 == static_cast<float>(1.0L - b2),
              "1 - beta");
        CHECK(a.lr == lh.lr && a.eps == lh.eps && a.wd == lh.weight_decay && a.beta1 == lh.beta1,
              "passed-through scalars");
    }
    dsm_destroy(ctx);
    // Global coefficients for n = 3 (not a power of two) and n = 4.
    for (int n : {3, 4}) {
        Problem Q({300}, n, 1, DSM_BASE_SGD_MOMENTUM);
        Buffers C(Q, false, true);
        CHECK(dsm_init(&Q.p, &C.b, &ctx) == DSM_OK, "init");
        const dsm_local_hparams sh = sgd_hp();
        for (int rule : {DSM_RULE_SIGN_MOMENTUM, DSM_RULE_GLOBAL_ADAMW}) {
            dsm_global_hparams g = glob_hp(DSM_SIGN_DET, rule);
            const int64_t t = rule == DSM_RULE_GLOBAL_ADAMW ? 77 : 4000000000LL;
            CHECK(dsm_local_step(ctx, -1, 1, &sh) == DSM_OK, "local");
            g_log.clear();
            CHECK(dsm_global_step(ctx, t, &g, 1) == DSM_OK, "global: %s", dsm_last_error(ctx));
            if (g_log.size() != 1) continue;
            const dsm::GlobalScalars& s = g_log[0].gs;
            const long double gam = g.gamma, eta = g.eta, b1 = g.beta1, b2 = g.beta2;
            CHECK(close_f32(s.c1, (1.0L - b1) / gam) && close_f32(s.c2, (1.0L - b2) / gam),
                  "c1 %.9g c2 %.9g", s.c1, s.c2);
            CHECK(close_f32(s.step, eta * gam), "eta gamma %.9g", s.step);
            CHECK(s.n == n && s.n_f == static_cast<float>(n) && s.n_pow2 == ((n & (n - 1)) == 0),
                  "worker count");
            CHECK(s.t == static_cast<uint32_t>(t) && s.rule == rule && s.lam == g.lambda, "t, rule");
            CHECK(g_log[0].v == C.b.v, "v passed");
            if (rule == DSM_RULE_GLOBAL_ADAMW) {
                CHECK(close_f32(s.bc1, 1.0L - std::pow(b1, static_cast<long double>(t + 1))) &&
                          close_f32(s.bc2, 1.0L - std::pow(b2, static_cast<long double>(t + 1))),
                      "Global AdamW bias corrections");
                CHECK(close_f32(s.inv_gamma, 1.0L / gam), "1/gamma");
            }
        }
        dsm_destroy(ctx);
    }
}

void check_hyperparameter_errors() {
    Problem P({100}, 2, 2, DSM_BASE_ADAMW);
    Buffers B(P, true, false);
    dsm_ctx* ctx = nullptr;
    CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init");
    g_log.clear();
    const float nan = std::nanf("");
    const float bad_lr[] = {0.0f, -1.0f, nan, INFINITY};
    for (float v : bad_lr) {
        dsm_local_hparams h = adam_hp();
        h.lr = v;
        CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_ERR_INVALID_ARG, "lr %g", v);
    }
    const float bad_beta[] = {-0.1f, 1.5f, nan, 1.0f};
    for (float v : bad_beta) {
        dsm_local_hparams h = adam_hp();
        h.beta1 = v;
        CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_ERR_INVALID_ARG, "beta1 %g", v);
        h = adam_hp();
        h.beta2 = v;
        CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_ERR_INVALID_ARG, "beta2 %g", v);
    }
    dsm_local_hparams h = adam_hp();
    h.eps = -1e-8f;
    CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_ERR_INVALID_ARG, "eps < 0");
    h = adam_hp();
    h.weight_decay = nan;
    CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_ERR_INVALID_ARG, "weight decay NaN");
    h = adam_hp();
    CHECK(dsm_local_step(ctx, -1, 0, &h) == DSM_ERR_INVALID_ARG, "step 0");
    CHECK(dsm_local_step(ctx, 2, 1, &h) == DSM_ERR_INVALID_ARG, "worker n");
    CHECK(dsm_local_step(ctx, -2, 1, &h) == DSM_ERR_INVALID_ARG, "worker -2");
    CHECK(dsm_local_step(ctx, -1, 1, nullptr) == DSM_ERR_INVALID_ARG, "NULL hparams");
    CHECK(g_log.empty(), "no launch after rejected local steps");
    CHECK(std::strlen(dsm_last_error(ctx)) > 0, "context error text");
    CHECK(dsm_local_step(ctx, -1, 1, &h) == DSM_OK, "step 1");
    CHECK(dsm_local_step(ctx, -1, 2, &h) == DSM_OK, "step 2");
    g_log.clear();
    struct {
        int field;
        float value;
    } bad_global[] = {{0, 0.0f}, {0, nan}, {1, -1.0f}, {2, 1.01f}, {3, -0.5f}, {4, -1.0f}, {4, INFINITY}};
    for (const auto& b : bad_global) {
        dsm_global_hparams g = glob_hp();
        float* f[] = {&g.gamma, &g.eta, &g.beta1, &g.beta2, &g.lambda};
        *f[b.field] = b.value;
        CHECK(dsm_global_step(ctx, 0, &g, 1) == DSM_ERR_INVALID_ARG, "global field %d = %g",
              b.field, b.value);
    }
    dsm_global_hparams g = glob_hp();
    g.mode = 3;
    CHECK(dsm_global_step(ctx, 0, &g, 1) == DSM_ERR_INVALID_ARG, "mode 3");
    g = glob_hp();
    g.rule = 4;
    CHECK(dsm_global_step(ctx, 0, &g, 1) == DSM_ERR_INVALID_ARG, "rule 4");
    g = glob_hp();
    CHECK(dsm_global_step(ctx, -1, &g, 1) == DSM_ERR_INVALID_ARG, "t < 0");
    CHECK(dsm_global_step(ctx, int64_t(1) << 32, &g, 1) == DSM_ERR_INVALID_ARG, "t = 2^32");
    CHECK(dsm_global_step(ctx, 0, nullptr, 1) == DSM_ERR_INVALID_ARG, "NULL global hparams");
    CHECK(g_log.empty(), "no launch after rejected global steps");
    CHECK(dsm_global_step(ctx, (int64_t(1) << 32) - 1, &g, 1) == DSM_OK, "largest t");
    CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
    // Calls on a NULL context.
    CHECK(dsm_local_step(nullptr, -1, 1, &h) == DSM_ERR_INVALID_ARG, "NULL ctx local");
    CHECK(dsm_global_step(nullptr, 0, &g, 1) == DSM_ERR_INVALID_ARG, "NULL ctx global");
    CHECK(dsm_round_end(nullptr, 1, &h, 0, &g, 1) == DSM_ERR_INVALID_ARG, "NULL ctx round end");
    CHECK(dsm_sync(nullptr) == DSM_ERR_INVALID_ARG, "NULL ctx sync");
    CHECK(dsm_read_bounds(nullptr, nullptr, 0) == DSM_ERR_INVALID_ARG, "NULL ctx bounds");
    CHECK(dsm_destroy(nullptr) == DSM_OK, "NULL ctx destroy");
}

void check_test_philox_args() {
    uint32_t* out = static_cast<uint32_t*>(std::aligned_alloc(256, 256));
    g_log.clear();
    CHECK(dsm_test_philox(1, 0, 0, 0, 16, out, nullptr) == DSM_OK, "valid");
    CHECK(dsm_test_philox(1, 0, 0, (int64_t(1) << 32) - 16, 16, out, nullptr) == DSM_OK,
          "last counter");
    CHECK(dsm_test_philox(1, 0, 0, (int64_t(1) << 32) - 15, 16, out, nullptr) == DSM_ERR_INVALID_ARG,
          "counter overflow");
    CHECK(dsm_test_philox(1, 0, -1, 0, 16, out, nullptr) == DSM_ERR_INVALID_ARG, "t < 0");
    CHECK(dsm_test_philox(1, 0, 0, 0, (int64_t(1) << 30) + 1, out, nullptr) == DSM_ERR_INVALID_ARG,
          "count above 2^30");
    CHECK(dsm_test_philox(1, 0, 0, 0, 16, out + 0, nullptr) == DSM_OK, "aligned");
    CHECK(dsm_test_philox(1, 0, 0, 0, 16,
                          reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(out) + 2),
                          nullptr) == DSM_ERR_INVALID_ARG,
          "misaligned output");
    CHECK(g_log.size() == 3, "three accepted calls launched, got %zu", g_log.size());
    g_devices = 0;
    CHECK(dsm_test_philox(1, 0, 0, 0, 16, out, nullptr) == DSM_ERR_HIP, "no device");
    g_devices = 1;
    std::free(out);
}

// The streaming diagnostic: whole pieces only, aligned buffers, the word
// array for reads, one launch of n_elems / DSM_PIECE_ELEMS work-groups.
void check_test_stream_args() {
    float* buf = static_cast<float*>(std::aligned_alloc(256, 4096 * 4));
    uint32_t* words = static_cast<uint32_t*>(std::aligned_alloc(256, 256));
    g_log.clear();
    CHECK(dsm_test_stream(DSM_STREAM_READ, buf, 4096, words, 0u, nullptr) == DSM_OK, "read");
    CHECK(g_log.size() == 1 && g_log[0].kind == "stream_read" && g_log[0].x == buf &&
              g_log[0].n_chunks == 4 && g_log[0].bounds == words,
          "read launch arguments");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf, 2048, nullptr, 0x3F800000u, nullptr) == DSM_OK, "write");
    CHECK(g_log.size() == 2 && g_log[1].kind == "stream_write" && g_log[1].n_chunks == 2,
          "write launch arguments");
    CHECK(dsm_test_stream(DSM_STREAM_READ, buf, 0, nullptr, 0u, nullptr) == DSM_OK, "empty");
    const int32_t bad_kind = 2;
    CHECK(dsm_test_stream(bad_kind, buf, 1024, words, 0u, nullptr) == DSM_ERR_INVALID_ARG,
          "unknown kind");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf, 1000, nullptr, 0u, nullptr) ==
              DSM_ERR_INVALID_ARG,
          "partial piece");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf, -1024, nullptr, 0u, nullptr) ==
              DSM_ERR_INVALID_ARG,
          "negative size");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf, (int64_t(1) << 24) * DSM_PIECE_ELEMS, nullptr,
                          0.f, nullptr) == DSM_ERR_INVALID_ARG,
          "beyond one grid dimension");
    CHECK(dsm_test_stream(DSM_STREAM_READ, buf, 1024, nullptr, 0u, nullptr) == DSM_ERR_INVALID_ARG,
          "read without words");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf + 1, 1024, nullptr, 0u, nullptr) ==
              DSM_ERR_INVALID_ARG,
          "misaligned buffer");
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, nullptr, 1024, nullptr, 0u, nullptr) ==
              DSM_ERR_INVALID_ARG,
          "NULL buffer");
    CHECK(dsm_test_stream(DSM_STREAM_READ, buf, 1024,
                          reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(words) + 2), 0u,
                          nullptr) == DSM_ERR_INVALID_ARG,
          "misaligned words");
    CHECK(g_log.size() == 3, "three accepted calls launched, got %zu", g_log.size());
    g_devices = 0;
    CHECK(dsm_test_stream(DSM_STREAM_WRITE, buf, 1024, nullptr, 0u, nullptr) == DSM_ERR_HIP,
          "no device");
    g_devices = 1;
    std::free(buf);
    std::free(words);
}

}  // namespace

// A split randomized global step passes the workspace's bound words, also
// for a problem with an empty tensor and for one with no chunks at all.
void check_global_rand_args() {
    for (const auto& shape : {std::vector<int64_t>{100, 16385, 0, 7}, std::vector<int64_t>{0, 0}}) {
        Problem P(shape, 2, 1, DSM_BASE_SGD_MOMENTUM);
        Buffers B(P, true, false);
        dsm_ctx* ctx = nullptr;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "init: %s", dsm_last_error(nullptr));
        const dsm_local_hparams sh = sgd_hp();
        CHECK(dsm_local_step(ctx, -1, 1, &sh) == DSM_OK, "local");
        const dsm_global_hparams gr = glob_hp(DSM_SIGN_RAND_ZERO);
        g_log.clear();
        CHECK(dsm_global_step(ctx, 5, &gr, 0) == DSM_OK, "randomized global: %s",
              dsm_last_error(ctx));
        CHECK(g_log.size() == 1, "one randomized launch, got %zu", g_log.size());
        if (g_log.size() == 1) {
            const Launch& l = g_log[0];
            CHECK(l.kind == "global_rand" && !l.broadcast && l.u == B.b.u_scratch &&
                      l.n_tensors == static_cast<int>(shape.size()),
                  "randomized launch arguments");
            check_bound_words(P, B, l.bounds, l.chunk0, l.piece_max, "global step");
        }
        CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
    }
}

// Blocked layouts: every work-group piece of every chunk lies inside one
// block, and (buffer, copy, element) -> slot covers each tensor element of each
// copy of each blocked buffer exactly once inside the allocation (n * d_pad
// for blocked replicas; B * n * d_pad for the replicas and their state), for
// random problems.
void check_blocked_addressing(int layout) {
    std::mt19937_64 rng(777 + layout);
    const int64_t piece = dsm::kPieceElems;
    const bool state = layout == DSM_REPLICAS_STATE_BLOCKED;
    for (int iter = 0; iter < 200; ++iter) {
        const int nt = 1 + static_cast<int>(rng() % 12);
        std::vector<int64_t> ne(nt);
        for (auto& v : ne) v = (rng() % 4 == 0) ? static_cast<int64_t>(rng() % 70000) : 1 + rng() % 3000;
        const int n = 1 + static_cast<int>(rng() % 9);
        const int base = state ? static_cast<int>(rng() % 2) : DSM_BASE_SGD_MOMENTUM;
        Problem P(ne, n, 2, base, {}, layout);
        Buffers B(P, false, false);
        const int64_t block = state ? 4096 : 16384;
        const int64_t shift = state ? 12 : 14;
        CHECK(B.arena % block == 0, "iter %d: blocked arena %lld not whole blocks", iter,
              static_cast<long long>(B.arena));
        dsm_ctx* ctx = nullptr;
        g_log.clear();
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "iter %d: init: %s", iter, dsm_last_error(nullptr));
        if (g_log.empty()) {
            dsm_destroy(ctx);
            continue;
        }
        const Launch& l = g_log[0];
        CHECK(same_layout(l.rl, B.rep), "iter %d: init layout", iter);
        // The blocked buffers and their offsets from the first one.
        std::vector<std::pair<dsm::RepLayout, int64_t>> bufs = {{l.rl, 0}};
        if (state) {
            CHECK(same_state(l.ml, B.rep), "iter %d: state layouts", iter);
            bufs.push_back({l.ml.g, B.b.g_rep - B.b.x_rep});
            bufs.push_back({l.ml.s1, B.b.s1_rep - B.b.x_rep});
            if (base == DSM_BASE_ADAMW) bufs.push_back({l.ml.s2, B.b.s2_rep - B.b.x_rep});
        }
        const int64_t total = static_cast<int64_t>(bufs.size()) * n * B.arena;
        const auto* c = static_cast<const dsm::Chunk*>(B.b.workspace);
        std::vector<uint8_t> seen(static_cast<size_t>(total), 0);
        bool ok_piece = true, ok_slot = true;
        for (int64_t k = 0; k < l.n_chunks; ++k) {
            for (int64_t e0 = c[k].off; e0 < c[k].off + c[k].len; e0 += piece) {
                const int64_t e1 = std::min<int64_t>(e0 + piece, c[k].off + c[k].len) - 1;
                ok_piece &= (e0 >> shift) == (e1 >> shift);
            }
            for (const auto& [L, off] : bufs) {
                for (int i = 0; i < n; ++i) {
                    for (int64_t e = c[k].off; e < c[k].off + c[k].len; ++e) {
                        const int64_t idx = off + rep_element(L, i, e);
                        if (idx < 0 || idx >= total || seen[idx]) {
                            ok_slot = false;
                        } else {
                            seen[idx] = 1;
                            // A piece's base plus the in-piece offset is the same slot.
                            const int64_t pb = c[k].off + ((e - c[k].off) / piece) * piece;
                            ok_slot &= off + rep_element(L, i, pb) + (e - pb) == idx;
                        }
                    }
                }
            }
        }
        CHECK(ok_piece, "iter %d: a piece crosses a block", iter);
        CHECK(ok_slot, "iter %d: slots overlap, leave the allocation or break within a piece", iter);
        CHECK(dsm_destroy(ctx) == DSM_OK, "destroy");
    }
    // The state-blocked layout refuses buffers that are not one allocation in
    // its order.
    if (state) {
        Problem P({5000, 7}, 3, 2, DSM_BASE_ADAMW, {}, layout);
        Buffers B(P, false, false);
        dsm_ctx* ctx = nullptr;
        float* keep = B.b.s2_rep;
        B.b.s2_rep = B.b.s1_rep;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_ERR_INVALID_ARG && ctx == nullptr,
              "state-blocked buffers out of order");
        CHECK(std::strstr(dsm_last_error(nullptr), "state-blocked") != nullptr, "order message");
        B.b.s2_rep = keep;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "state-blocked in order");
        dsm_destroy(ctx);
    }
}

// dsm_init_static: the workspace and the u staging come from the static
// scratch (the caller's are ignored), the size limit, one live context per
// device, and the device released by dsm_destroy.
void check_init_static() {
    Problem P({100, 16385, 7}, 3, 2, DSM_BASE_ADAMW, {1, 1, 0}, DSM_REPLICAS_BLOCKED);
    Buffers B(P, false, false);            // no u_scratch of its own
    B.b.workspace = nullptr;               // and no workspace
    B.b.workspace_bytes = 0;
    int64_t arena = 0, ws = 0;
    CHECK(dsm_layout(&P.p, &arena, nullptr, &ws) == DSM_OK, "layout");
    dsm_ctx* a = nullptr;
    g_log.clear();
    CHECK(dsm_init_static(&P.p, &B.b, &a) == DSM_OK && a != nullptr, "static init: %s",
          dsm_last_error(nullptr));
    CHECK(g_log.size() == 1 && g_log[0].kind == "init" && g_log[0].chunks == g_scratch &&
              same_layout(g_log[0].rl, B.rep),
          "the chunk table lives in the static scratch");
    const auto* c = static_cast<const dsm::Chunk*>(g_scratch);
    CHECK(c[0].tensor == 0 && c[0].len == 100 && c[1].tensor == 1 && c[1].len == 16384,
          "chunk table uploaded into the scratch");
    // A second static context on the same device is refused; on another
    // device it is allowed.
    dsm_ctx* b2 = nullptr;
    CHECK(dsm_init_static(&P.p, &B.b, &b2) == DSM_ERR_STATE && b2 == nullptr,
          "second static context on device 0");
    CHECK(std::strstr(dsm_last_error(nullptr), "dsm_init_static") != nullptr, "busy message");
    // The randomized global step takes u from the scratch, after the workspace.
    const dsm_local_hparams lh = adam_hp();
    for (int k = 0; k < 2; ++k) CHECK(dsm_local_step(a, -1, k + 1, &lh) == DSM_OK, "local");
    const dsm_global_hparams gr = glob_hp(DSM_SIGN_RAND_FLIP);
    g_log.clear();
    CHECK(dsm_global_step(a, 0, &gr, 1) == DSM_OK, "randomized step: %s", dsm_last_error(a));
    if (g_log.size() == 1) {
        const char* base = static_cast<const char*>(g_scratch);
        CHECK(reinterpret_cast<const char*>(g_log[0].u) == base + round_up(ws, 256),
              "u staging follows the workspace in the scratch");
        CHECK(reinterpret_cast<const char*>(g_log[0].u) + arena * 4 <=
                  base + dsm::kStaticScratchBytes,
              "u staging inside the scratch");
        B.b.workspace = g_scratch;         // where the words must be
        B.b.workspace_bytes = ws;
        check_bound_words(P, B, g_log[0].bounds, g_log[0].chunk0, g_log[0].piece_max, "static");
    }
    CHECK(dsm_destroy(a) == DSM_OK, "destroy");
    // Released: the device's scratch can be taken again, by a smaller problem.
    Problem Q({5000}, 2, 1, DSM_BASE_SGD_MOMENTUM);
    Buffers C(Q, true, false);
    dsm_ctx* q = nullptr;
    CHECK(dsm_init_static(&Q.p, &C.b, &q) == DSM_OK, "static init after destroy");
    CHECK(dsm_destroy(q) == DSM_OK, "destroy");
    // Too large for the scratch: refused with the sizes, nothing launched.
    const int64_t big = (dsm::kStaticScratchBytes / 4) + 1;
    Problem R_({big}, 1, 1, DSM_BASE_SGD_MOMENTUM);
    std::vector<uint8_t> dummy(512);
    dsm_buffers rb{};
    rb.x = rb.m = rb.x_rep = rb.g_rep = rb.s1_rep = reinterpret_cast<float*>(
        reinterpret_cast<uintptr_t>(dummy.data() + 255) & ~uintptr_t(255));
    g_log.clear();
    dsm_ctx* r = nullptr;
    CHECK(dsm_init_static(&R_.p, &rb, &r) == DSM_ERR_INVALID_ARG && r == nullptr,
          "problem beyond the static scratch");
    CHECK(std::strstr(dsm_last_error(nullptr), "static scratch") != nullptr, "limit message");
    CHECK(g_log.empty(), "nothing launched for a rejected static context");
    // Device 1: its own scratch slot, independent of device 0's.
    g_device = 1;
    dsm_ctx* d1 = nullptr;
    dsm_ctx* d0 = nullptr;
    CHECK(dsm_init_static(&Q.p, &C.b, &d1) == DSM_OK, "static context on device 1");
    g_device = 0;
    CHECK(dsm_init_static(&Q.p, &C.b, &d0) == DSM_OK, "and one on device 0");
    CHECK(dsm_destroy(d1) == DSM_OK && dsm_destroy(d0) == DSM_OK, "destroy both");
    std::free(g_scratch);
    g_scratch = nullptr;
}

// The worker-interleaved local-step order keeps the whole pieces x workers row
// in one grid dimension of fewer than 2^32 threads, or falls back to the
// worker-by-worker grid.
void check_local_map() {
    using dsm::kBlockThreads;
    using dsm::kInterleaveWorkers;
    using dsm::kSplit;
    const int64_t limit = (int64_t(1) << 32) / kBlockThreads;  // work-groups per row
    for (int base : {0, 1, 2}) {
        const int il = base | kInterleaveWorkers;
        for (int n : {1, 2, 3, 8, 64}) {
            // The largest chunk count whose row fits, and one more.
            const int64_t fit = (limit - 1) / (int64_t(kSplit) * n);
            CHECK(dsm::local_map(fit, n, il) == il, "row of %lld chunks x %d workers fits",
                  static_cast<long long>(fit), n);
            CHECK(fit * kSplit * n * kBlockThreads < (int64_t(1) << 32), "fit really fits");
            const int64_t over = fit + 1;
            CHECK(over * kSplit * n * kBlockThreads >= (int64_t(1) << 32) ?
                      dsm::local_map(over, n, il) == base : dsm::local_map(over, n, il) == il,
                  "row of %lld chunks x %d workers", static_cast<long long>(over), n);
            CHECK(dsm::local_map(over, n, base) == base, "no interleave bit, no change");
            CHECK(dsm::local_map(1LL << 40, n, il) == base, "huge row falls back");
        }
    }
    // The state-blocked layout's default local map interleaves the workers.
    CHECK(dsm::kMapsByLayout[DSM_REPLICAS_STATE_BLOCKED].local & kInterleaveWorkers,
          "state-blocked local steps interleave workers");
}

// Contexts share no state but the static-scratch slot of each device and the
// per-thread last error.  Four threads each drive their own context through
// rounds of Algorithm 1 at once (both bases, all three replica layouts), each
// provoking an error whose text must come back to it and not to another
// thread; three more take turns on the device's one static-scratch slot, which
// must never hold two live contexts.
void check_threads() {
    std::atomic<int> static_alive{0}, static_max{0}, static_wins{0};
    auto own_context = [&](int seed) {
        const int base = seed % 2 ? DSM_BASE_SGD_MOMENTUM : DSM_BASE_ADAMW;
        Problem P({1000 + 17 * seed, 3000, 64}, 2, 3, base, {}, seed % 3);
        Buffers B(P, true, false);
        dsm_ctx* ctx = nullptr;
        CHECK(dsm_init(&P.p, &B.b, &ctx) == DSM_OK, "thread %d: init", seed);
        if (!ctx) return;
        const dsm_local_hparams lh = base == DSM_BASE_ADAMW ? adam_hp() : sgd_hp();
        for (int t = 0; t < 4; ++t) {
            const dsm_global_hparams gh = glob_hp(t % 2 ? DSM_SIGN_RAND_FLIP : DSM_SIGN_DET);
            for (int k = 0; k < 3; ++k)
                CHECK(dsm_local_step(ctx, -1, 3 * t + k + 1, &lh) == DSM_OK, "thread %d: local",
                      seed);
            CHECK(dsm_global_step(ctx, t, &gh, 1) == DSM_OK, "thread %d: global", seed);
        }
        const int bad = 50 + seed;
        CHECK(dsm_local_step(ctx, bad, 1, &lh) == DSM_ERR_INVALID_ARG, "thread %d: bad worker",
              seed);
        char want[32];
        std::snprintf(want, sizeof want, "got %d", bad);
        const std::string mine = dsm_last_error(nullptr);
        CHECK(mine.find(want) != std::string::npos, "thread %d: its own error text, got '%s'", seed,
              mine.c_str());
        CHECK(std::string(dsm_last_error(ctx)).find(want) != std::string::npos,
              "thread %d: the context's error text", seed);
        CHECK(dsm_destroy(ctx) == DSM_OK, "thread %d: destroy", seed);
    };
    auto static_turns = [&](int seed) {
        Problem P({2000 + seed, 40}, 2, 1, DSM_BASE_SGD_MOMENTUM);
        Buffers B(P, false, false);
        dsm_buffers b = B.b;
        b.workspace = nullptr;
        b.workspace_bytes = 0;
        b.u_scratch = nullptr;
        const dsm_local_hparams lh = sgd_hp();
        for (int it = 0; it < 200; ++it) {
            dsm_ctx* ctx = nullptr;
            const dsm_status st = dsm_init_static(&P.p, &b, &ctx);
            if (st == DSM_ERR_STATE) {
                std::this_thread::yield();
                continue;
            }
            CHECK(st == DSM_OK, "static thread %d: init (%d)", seed, static_cast<int>(st));
            if (st != DSM_OK) return;
            const int alive = ++static_alive;
            int prev = static_max.load();
            while (alive > prev && !static_max.compare_exchange_weak(prev, alive)) {
            }
            ++static_wins;
            CHECK(dsm_local_step(ctx, -1, 1, &lh) == DSM_OK, "static thread %d: local", seed);
            --static_alive;  // before the slot is released, so no later owner overlaps it
            CHECK(dsm_destroy(ctx) == DSM_OK, "static thread %d: destroy", seed);
        }
    };
    std::vector<std::thread> threads;
    for (int i = 0; i < 4; ++i) threads.emplace_back(own_context, i);
    for (int i = 0; i < 3; ++i) threads.emplace_back(static_turns, i);
    for (auto& t : threads) t.join();
    CHECK(static_max.load() == 1, "static contexts alive at once: %d", static_max.load());
    CHECK(static_wins.load() > 0, "no thread got the static scratch");
}

int main(int argc, char** argv) {
    if (argc == 2 && std::strcmp(argv[1], "threads") == 0) {
        check_threads();
        if (g_failures) {
            std::fprintf(stderr, "%d of %d checks failed\n", g_failures.load(), g_checks.load());
            return 1;
        }
        std::printf("all checks passed (%d)\n", g_checks.load());
        return 0;
    }
    check_local_map();
    check_layout_fuzz();
    check_init_and_chunks();
    check_init_rejections();
    check_init_static();
    check_blocked_addressing(DSM_REPLICAS_BLOCKED);
    check_blocked_addressing(DSM_REPLICAS_STATE_BLOCKED);
    for (int layout : {DSM_REPLICAS_CONTIGUOUS, DSM_REPLICAS_BLOCKED, DSM_REPLICAS_STATE_BLOCKED}) {
        check_state_machine_adamw(layout);
        check_state_machine_sgd_h1(layout);
        check_local_from_x(layout);
    }
    check_coefficients();
    check_global_rand_args();
    check_hyperparameter_errors();
    check_test_philox_args();
    check_test_stream_args();
    check_threads();
    if (g_failures) {
        std::fprintf(stderr, "%d of %d checks failed\n", g_failures.load(), g_checks.load());
        return 1;
    }
    std::printf("all checks passed (%d)\n", g_checks.load());
    return 0;
}
