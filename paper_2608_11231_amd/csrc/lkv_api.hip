// C ABI of liblkv.so (declared in include/lkv.h): host-side validation,
// launch-geometry selection and dispatch to the gfx950 kernels.
#include <stdlib.h>

#include <atomic>
#include <mutex>

#include "decode_kernels.h"
#include "diag_kernels.h"
#include "gather_kernels.h"
#include "pool_kernels.h"
#include "sp_kernels.h"
#include "init_kernels.h"
#include "lkv.h"
#include "chunk_kernel.h"

using namespace lkv;

namespace {

thread_local int g_last_hip = 0;
// polls of the chunk kernels' bounded stager -> solver wait (lkv_set_wait_limit)
constexpr int32_t kDefaultWaitLimit = 1 << 14;
std::atomic<int32_t> g_wait_limit{kDefaultWaitLimit};

lkv_status hip_status(hipError_t e) {
    if (e == hipSuccess) return LKV_OK;
    g_last_hip = (int)e;
    return LKV_E_HIP;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

lkv_status check_layer(const lkv_layer* L) {
    if (!L) return LKV_E_NULL;
    if (L->family != LKV_GDN && L->family != LKV_SSD) return LKV_E_SHAPE;
    if (L->h_qk < 1 || L->h_v < 1 || L->h_v % L->h_qk != 0) return LKV_E_SHAPE;
    if (L->dk < 1 || L->dv < 1 || L->chunk < 1) return LKV_E_SHAPE;
    if (L->io_dtype != LKV_F32 && L->io_dtype != LKV_BF16) return LKV_E_DTYPE;
    if (L->gate_dtype != LKV_F32 && L->gate_dtype != LKV_BF16) return LKV_E_DTYPE;
    if (L->family == LKV_SSD && L->gate_dtype != LKV_F32) return LKV_E_DTYPE;
    if (L->dk != 16 && L->dk != 32 && L->dk != 64 && L->dk != 128) return LKV_E_UNSUPPORTED;
    if (L->dv % 16 != 0 || L->dv > 512) return LKV_E_UNSUPPORTED;
    if (L->chunk != 16 && L->chunk != 64) return LKV_E_UNSUPPORTED;
    // fp32 q/k/v double the staged tiles: supported up to dk = 64
    if (L->io_dtype == LKV_F32 && L->dk > 64) return LKV_E_UNSUPPORTED;
    return LKV_OK;
}

int env_int(const char* name, int dflt) {
    const char* s = getenv(name);
    return s ? atoi(s) : dflt;
}

// State-row waves per workgroup for the chunk kernels (16*nb rows per
// workgroup; every workgroup also runs 4 waves for the state-independent
// work).  More rows per workgroup share that work; fewer give more workgroups.
// Pick the largest nb that fits LDS and still fills the 256 CUs.
int pick_nw(int fam, int dk, int chunk, bool f32io, int64_t pairs, int rows, int rows2, bool summary) {
    int forced = env_int("LKV_SCAN_NB", 0);
    int fallback = 0;
    for (int nb = summary ? 8 : 4; nb >= 1; nb >>= 1) {
        if (rows % (16 * nb) || (rows2 && rows2 % (16 * nb))) continue;
        const size_t lds = scan_lds_bytes(fam, dk, chunk, f32io, nb, summary);
        if (lds == 0 || lds > 160 * 1024) continue;
        if (forced) {
            if (nb == forced) return nb;
            continue;
        }
        if (!fallback) fallback = nb;
        const int64_t units = pairs * ((rows + (rows2 ? rows2 : 0)) / (16 * nb));
        if (units >= 240) return nb;
        fallback = nb;
    }
    return fallback;
}

lkv_status check_tokens(const lkv_layer* L, const lkv_tokens* T, bool need_q, bool need_v = true,
                        bool need_k = true) {
    if (!T) return LKV_E_NULL;
    if (T->n_seq < 0 || T->n_tok < 0) return LKV_E_SHAPE;
    if (T->n_seq > 0 && !T->cu) return LKV_E_NULL;
    if (T->n_tok > 0) {
        if ((need_k && !T->k) || (need_v && !T->v) || !T->g) return LKV_E_NULL;
        if (need_q && !T->q) return LKV_E_NULL;
        if (L->family == LKV_GDN && !T->beta) return LKV_E_NULL;
        if ((need_k && !aligned16(T->k)) || (need_v && !aligned16(T->v)) || (need_q && !aligned16(T->q)))
            return LKV_E_ALIGN;
    }
    if (L->family == LKV_SSD && T->n_seq > 0 && !T->A) return LKV_E_NULL;
    if (T->n_tok > INT64_C(1) << 40) return LKV_E_SHAPE;
    return LKV_OK;
}

ScanArgs base_args(const lkv_layer* L, const lkv_tokens* T) {
    ScanArgs a = {};
    a.cu = T->cu;
    a.n_seq = T->n_seq;
    a.n_tok = T->n_tok;
    a.q = T->q;
    a.k = T->k;
    a.v = T->v;
    a.g = T->g;
    a.beta = T->beta;
    a.A = T->A;
    a.h_qk = L->h_qk;
    a.h_v = L->h_v;
    a.dv = L->dv;
    a.gate_bf16 = L->gate_dtype == LKV_BF16;
    a.scale = 1.f;
    a.wait_limit = g_wait_limit.load(std::memory_order_relaxed);
    return a;
}

// Mamba-2 scans and block summaries can run on ssd_scan_kernel where it
// covers the shapes (bf16 io, 64-token chunks, dk >= 32, dv a multiple of 64):
// LKV_SSD_SCAN_KERNEL=1 selects it, otherwise the shared chunk kernel runs
// (the two give identical bits).
bool use_ssd_scan(const lkv_layer* L) {
    return L->family == LKV_SSD && env_int("LKV_SSD_SCAN_KERNEL", 0) == 1 &&
           ssd_scan_supported(L->dk, L->chunk, L->io_dtype == LKV_F32, L->dv);
}

// The sequence-parallel Mamba-2 scan as one pass over the pieces plus an
// output correction, on the same shapes; LKV_SSD_SP_CORRECT=0 selects the
// summary / composition / rescan form shared with Gated DeltaNet.
bool use_ssd_sp(const lkv_layer* L) {
    return L->family == LKV_SSD && env_int("LKV_SSD_SP_CORRECT", 1) == 1 &&
           ssd_scan_supported(L->dk, L->chunk, L->io_dtype == LKV_F32, L->dv);
}

lkv_status ssd_scan(const lkv_layer* L, ScanArgs a, int64_t pairs, hipStream_t st) {
    const int64_t units = pairs * (L->dv / 64);
    if (units >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    a.tiles_b = L->dv / 64;
    a.tiles_m = 0;
    a.nb = 4;
    a.n_units = (int32_t)units;
    return hip_status(launch_ssd_scan(L->dk, a, st));
}

hipError_t launch_scan(const lkv_layer* L, const ScanArgs& a, hipStream_t st) {
    const bool f32io = L->io_dtype == LKV_F32;
    return L->family == LKV_GDN ? launch_scan_gdn(L->dk, L->chunk, f32io, a, st)
                                : launch_scan_ssd(L->dk, L->chunk, f32io, a, st);
}

lkv_status chunk_scan(const lkv_layer* L, const lkv_tokens* T, float scale, const float* S_init, void* out,
                      float* S_final, void* stream, const int32_t* src = nullptr, int32_t n_src = 0,
                      bool init_bf16 = false) {
    lkv_status s = check_tokens(L, T, out != nullptr);
    if (s != LKV_OK) return s;
    if ((S_init && !aligned16(S_init)) || (S_final && !aligned16(S_final))) return LKV_E_ALIGN;
    if (T->n_seq == 0) return LKV_OK;
    if (!out && !S_final) return LKV_OK;
    const bool f32io = L->io_dtype == LKV_F32;
    const int64_t pairs = (int64_t)T->n_seq * L->h_v;
    ScanArgs a = base_args(L, T);
    a.scale = scale;
    a.S_init = S_init;
    a.src = src;
    a.n_src = n_src;
    a.init_bf16 = init_bf16 ? 1 : 0;
    a.out = out;
    a.S_final = S_final;
    a.summary = 0;
    if (use_ssd_scan(L)) return ssd_scan(L, a, pairs, (hipStream_t)stream);
    const int nw = pick_nw(L->family, L->dk, L->chunk, f32io, pairs, L->dv, 0, false);
    if (nw == 0) return LKV_E_UNSUPPORTED;
    const int64_t units = pairs * (L->dv / (16 * nw));
    if (units >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    a.tiles_b = L->dv / (16 * nw);
    a.tiles_m = 0;
    a.nb = nw;
    a.n_units = (int32_t)units;
    return hip_status(launch_scan(L, a, (hipStream_t)stream));
}

lkv_status decode(const lkv_layer* L, int32_t n_req, const void* q, const void* k, const void* v,
                  const void* g, const void* beta, const float* A, float scale, float* S, void* o, void* stream) {
    if (n_req < 0) return LKV_E_SHAPE;
    if (n_req == 0) return LKV_OK;
    if (!q || !k || !v || !g || !S || (L->family == LKV_GDN && !beta)) return LKV_E_NULL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(S)) return LKV_E_ALIGN;
    if ((int64_t)n_req * L->h_v * (L->dv / 16) >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    DecodeArgs a = {};
    a.n_req = n_req;
    a.h_qk = L->h_qk;
    a.h_v = L->h_v;
    a.dv = L->dv;
    a.io_bf16 = L->io_dtype == LKV_BF16;
    a.gate_bf16 = L->gate_dtype == LKV_BF16;
    a.q = q;
    a.k = k;
    a.v = v;
    a.g = g;
    a.beta = beta;
    a.A = A;
    a.scale = scale;
    a.S = S;
    a.out = o;
    return hip_status(launch_decode(L->family == LKV_GDN ? 0 : 1, L->dk, a, (hipStream_t)stream));
}

lkv_status init_single(const lkv_layer* L, int32_t n_req, int32_t n_blk, const void* B_pool, bool bf16_pool,
                       const int32_t* src_blk, float* S_init, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (n_req < 0 || n_blk < 0) return LKV_E_SHAPE;
    if (n_req == 0) return LKV_OK;
    if (!src_blk || !S_init || (n_blk > 0 && !B_pool)) return LKV_E_NULL;
    if (!aligned16(S_init) || (B_pool && !aligned16(B_pool))) return LKV_E_ALIGN;
    const int64_t per_req = (int64_t)L->h_v * L->dv * L->dk;
    return hip_status(launch_init_single(n_req, n_blk, per_req, B_pool, bf16_pool, src_blk, S_init,
                                         (hipStream_t)stream));
}

lkv_status init_compose(const lkv_layer* L, int32_t n_req, int32_t n_blk, const void* B_pool, bool bf16_pool,
                        const float* M_pool, const int32_t* blk_ids, const int32_t* blk_cu, int32_t n_ids,
                        float* S_init, void* stream, float* S_steps = nullptr) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (n_req < 0 || n_blk < 0 || n_ids < 0) return LKV_E_SHAPE;
    if (n_req == 0) return LKV_OK;
    if (!blk_cu || !S_init || (n_ids > 0 && !blk_ids)) return LKV_E_NULL;
    if (n_blk > 0 && (!B_pool || !M_pool)) return LKV_E_NULL;
    if (!aligned16(S_init) || (B_pool && !aligned16(B_pool)) || (M_pool && !aligned16(M_pool)))
        return LKV_E_ALIGN;
    hipStream_t st = (hipStream_t)stream;
    if (L->family == LKV_SSD) {
        const int64_t per_head = (int64_t)L->dv * L->dk;
        return hip_status(launch_compose_ssd(n_req, n_blk, L->h_v, per_head, B_pool, bf16_pool, M_pool, blk_ids,
                                             blk_cu, n_ids, S_init, S_steps, st));
    }
    const int64_t pairs = (int64_t)n_req * L->h_v;
    // waves per workgroup: eight on 64 state rows (two per row tile, each
    // with half of the state's dk tiles) where dk >= 32 and dv allows, else
    // four, two or one of 16 rows each.  Each step stages the whole M in LDS;
    // the waves share that staging, and the step's latency -- not the number
    // of workgroups -- sets the time (at 8K, 64 four-wave workgroups compose
    // faster than 256 one-wave ones)
    int nw = env_int("LKV_COMPOSE_NW", 0);
    if (nw != 1 && nw != 2 && nw != 4 && nw != 8) nw = 8;
    if (nw == 8 && (L->dk < 32 || L->dv % 64)) nw = 4;
    while (nw > 1 && nw != 8 && L->dv % (16 * nw)) nw >>= 1;
    const int rows = nw == 8 ? 64 : 16 * nw;  // state rows per workgroup
    ComposeArgs a = {};
    a.B_pool = B_pool;
    a.bf16_pool = bf16_pool;
    a.M_pool = M_pool;
    a.blk_ids = blk_ids;
    a.blk_cu = blk_cu;
    a.n_ids = n_ids;
    a.n_blk = n_blk;
    a.h_v = L->h_v;
    a.dv = L->dv;
    a.S = S_init;
    a.S_steps = S_steps;
    a.nw = nw;
    a.tiles = L->dv / rows;
    const int64_t units = pairs * a.tiles;
    if (units >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    a.n_units = (int32_t)units;
    return hip_status(launch_compose_gdn(L->dk, a, st));
}

// Workspace of the sequence-parallel scan, each region 256-byte aligned:
// piece offsets, the composition's block ids and offsets, the block pools
// (every piece's end state from zero and transition, then one row per
// request holding its initial state), and every piece's start state.
struct SpLayout {
    size_t piece_cu, blk_ids, blk_cu, B, M, S_start, S_last, total;
};

SpLayout sp_layout(const lkv_layer* L, int64_t n_req, int64_t pieces) {
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    const int64_t n_seg = n_req * pieces;
    const size_t state = (size_t)L->h_v * L->dv * L->dk * 4;
    const size_t trans = L->family == LKV_GDN ? (size_t)L->h_v * L->dk * L->dk * 4 : (size_t)L->h_v * 4;
    SpLayout o{};
    size_t at = 0;
    o.piece_cu = at; at += up((size_t)(n_seg + 1) * 4);
    o.blk_ids = at;  at += up((size_t)n_req * (pieces + 1) * 4);
    o.blk_cu = at;   at += up((size_t)(n_req + 1) * 4);
    o.B = at;        at += up((size_t)(n_seg + n_req) * state);
    o.M = at;        at += up((size_t)(n_seg + n_req) * trans);
    o.S_start = at;  at += up((size_t)n_seg * state);
    o.S_last = at;   at += up((size_t)n_req * state);  // the final states when S_final is NULL
    o.total = at;
    return o;
}

lkv_status sp_check(const lkv_layer* L, int32_t n_req, int32_t pieces) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (n_req < 0 || pieces < 1 || pieces > 64) return LKV_E_SHAPE;
    if ((int64_t)n_req * (pieces + 1) >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    return LKV_OK;
}

lkv_status chunk_scan_sp(const lkv_layer* L, const lkv_tokens* T, float scale, const float* S_init, void* out,
                         float* S_final, int32_t pieces, char* ws, size_t ws_bytes, void* stream) {
    if (!T) return LKV_E_NULL;
    lkv_status s = sp_check(L, T->n_seq, pieces);
    if (s != LKV_OK) return s;
    s = check_tokens(L, T, out != nullptr);
    if (s != LKV_OK) return s;
    if ((S_init && !aligned16(S_init)) || (S_final && !aligned16(S_final))) return LKV_E_ALIGN;
    if (T->n_seq == 0 || (!out && !S_final)) return LKV_OK;
    const SpLayout ly = sp_layout(L, T->n_seq, pieces);
    if (!ws) return LKV_E_NULL;
    if (((uintptr_t)ws & 255u) != 0) return LKV_E_ALIGN;
    if (ws_bytes < ly.total) return LKV_E_SHAPE;
    hipStream_t st = (hipStream_t)stream;
    const int32_t n_req = T->n_seq, n_seg = n_req * pieces;
    int32_t* piece_cu = reinterpret_cast<int32_t*>(ws + ly.piece_cu);
    int32_t* blk_ids = reinterpret_cast<int32_t*>(ws + ly.blk_ids);
    int32_t* blk_cu = reinterpret_cast<int32_t*>(ws + ly.blk_cu);
    float* Bp = reinterpret_cast<float*>(ws + ly.B);
    float* Mp = reinterpret_cast<float*>(ws + ly.M);
    float* S_start = reinterpret_cast<float*>(ws + ly.S_start);
    float* S_last = S_final ? S_final : reinterpret_cast<float*>(ws + ly.S_last);
    const int64_t state = (int64_t)L->h_v * L->dv * L->dk;
    if (pieces > 1 && use_ssd_sp(L)) {
        // Mamba-2: the pieces scanned once, piece 0 from the initial state and
        // the others from zero, then their outputs corrected and the final
        // state composed (ssd_correct_kernel)
        const int tiles = L->dv / 64;
        const int64_t units = (int64_t)n_seg * L->h_v * tiles;
        if (units >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
        ScanArgs a = base_args(L, T);
        a.S_init = S_init;
        a.out = out;
        a.summary = 0;
        a.tiles_b = tiles;
        a.nb = 4;
        a.n_units = (int32_t)units;
        a.pieces = pieces;
        a.piece_B = Bp;
        a.piece_L = Mp;
        lkv_status e = hip_status(launch_ssd_scan(L->dk, a, st));
        if (e != LKV_OK) return e;
        SsdCorrectArgs c = {};
        c.cu = T->cu;
        c.n_seq = n_req;
        c.n_tok = T->n_tok;
        c.C = T->q;
        c.dt = reinterpret_cast<const float*>(T->g);
        c.A = T->A;
        c.h_qk = L->h_qk;
        c.h_v = L->h_v;
        c.dv = L->dv;
        c.pieces = pieces;
        c.piece_B = Bp;
        c.piece_L = Mp;
        c.y = out;
        c.S_final = S_final;
        c.tiles = tiles;
        // chunk slots: about one workgroup per CU, at most a piece's chunks
        // (ceil(ceil(n_tok / P) / CH) bounds them) and at most 8
        const int64_t max_chunks = ((T->n_tok + pieces - 1) / pieces + L->chunk - 1) / L->chunk;
        const int64_t base = (int64_t)n_req * (pieces - 1) * L->h_v * tiles;
        int64_t slots = (256 + base - 1) / base;
        if (slots > max_chunks) slots = max_chunks;
        if (env_int("LKV_SSD_CORRECT_SLOTS", 0) > 0) slots = env_int("LKV_SSD_CORRECT_SLOTS", 0);
        c.slots = (int32_t)(slots < 1 ? 1 : (slots > 8 ? 8 : slots));
        const int64_t cunits = (int64_t)n_req * (pieces - 1) * L->h_v * tiles * c.slots;
        if (cunits >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
        c.n_units = (int32_t)cunits;
        return hip_status(launch_ssd_correct(L->dk, c, st));
    }
    lkv_status e = hip_status(launch_sp_setup(T->cu, n_req, pieces, L->chunk, T->n_tok, piece_cu, blk_ids, blk_cu,
                                              S_init, Bp + (int64_t)n_seg * state, state, st));
    if (e != LKV_OK) return e;
    // every piece's (transition, state from zero): Eq. 5 per piece, one launch
    lkv_tokens Tp = *T;
    Tp.cu = piece_cu;
    Tp.n_seq = n_seg;
    Tp.q = nullptr;
    e = lkv_block_summary(L, &Tp, Bp, Mp, stream);
    if (e != LKV_OK) return e;
    // the pieces' start states and the final state: each request's initial
    // state composed with its pieces' pairs, the state after every piece kept
    e = init_compose(L, n_req, n_seg + n_req, Bp, false, Mp, blk_ids, blk_cu, n_req * (pieces + 1), S_last, stream,
                     S_start);
    if (e != LKV_OK || !out) return e;
    // the outputs: every piece scanned from its start state, all at once
    Tp.q = T->q;
    return chunk_scan(L, &Tp, L->family == LKV_GDN ? scale : 1.f, S_start, out, nullptr, stream);
}

// Scratch of the allocation-free sequence-parallel scan: one fixed array per
// GPU, in the library's device code, held until the process ends.  Host code
// never uses the array's name (on the host it is only a stand-in for the
// symbol): its device address is taken once per device with
// hipGetSymbolAddress, with that device current, and kept here.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

lkv_status scratch_for_current_device(char** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e);
    if (dev < 0 || dev >= kMaxDevices) return LKV_E_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e);
        if (!ptr) return LKV_E_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = reinterpret_cast<char*>(g_scratch_ptr[dev]);
    return LKV_OK;
}

}  // namespace

extern "C" {

int lkv_abi_version(void) { return LKV_ABI_VERSION; }

const char* lkv_status_string(lkv_status s) {
    switch (s) {
        case LKV_OK: return "ok";
        case LKV_E_NULL: return "a required pointer is NULL";
        case LKV_E_SHAPE: return "invalid or inconsistent size";
        case LKV_E_DTYPE: return "unsupported dtype";
        case LKV_E_ALIGN: return "tensor pointer not 16-byte aligned";
        case LKV_E_UNSUPPORTED: return "geometry not implemented by this build";
        case LKV_E_WORKSPACE: return "needs more scratch than the allocation-free variant's fixed 64 MiB per GPU";
        case LKV_E_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

int lkv_last_hip_error(void) { return g_last_hip; }

int32_t lkv_set_wait_limit(int32_t polls) {
    if (polls < 0) polls = kDefaultWaitLimit;
    return g_wait_limit.exchange(polls, std::memory_order_relaxed);
}

lkv_status lkv_block_summary(const lkv_layer* L, const lkv_tokens* T, float* B_out, float* M_out,
                             void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (!B_out && !M_out) return LKV_E_NULL;
    // transitions read no values: v may be NULL when B_out is; Mamba-2's
    // transitions read only dt (and A)
    s = check_tokens(L, T, false, B_out != nullptr, B_out != nullptr || L->family == LKV_GDN);
    if (s != LKV_OK) return s;
    if ((B_out && !aligned16(B_out)) || (M_out && !aligned16(M_out))) return LKV_E_ALIGN;
    if (T->n_seq == 0) return LKV_OK;
    const bool f32io = L->io_dtype == LKV_F32;
    const int64_t pairs = (int64_t)T->n_seq * L->h_v;
    const bool gdn_m = L->family == LKV_GDN && M_out;
    const int rows_b = B_out ? L->dv : 0;
    const int rows_m = gdn_m ? L->dk : 0;
    ScanArgs a = base_args(L, T);
    a.summary = 1;
    a.S_final = B_out;
    a.M_out = M_out;
    hipStream_t st = (hipStream_t)stream;
    if (L->family == LKV_SSD && !B_out) {
        // Lambda only: a segmented sum of the dt column, no state work
        if (pairs >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
        return hip_status(launch_ssd_lambda(T->cu, T->n_seq, T->n_tok, L->h_v, reinterpret_cast<const float*>(T->g),
                                            T->A, M_out, st));
    }
    if (use_ssd_scan(L)) return ssd_scan(L, a, pairs, st);
    const int nw = pick_nw(L->family, L->dk, L->chunk, f32io, pairs, rows_b ? rows_b : rows_m,
                           rows_b ? rows_m : 0, true);
    if (nw == 0) return LKV_E_UNSUPPORTED;
    a.nb = nw;
    a.tiles_b = rows_b / (16 * nw);
    a.tiles_m = rows_m / (16 * nw);
    const int64_t units = pairs * (a.tiles_b + a.tiles_m);
    if (units >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    a.n_units = (int32_t)units;
    return hip_status(launch_scan(L, a, st));
}

lkv_status lkv_init_single(const lkv_layer* L, int32_t n_req, int32_t n_blk, const float* B_pool,
                           const int32_t* src_blk, float* S_init, void* stream) {
    return init_single(L, n_req, n_blk, B_pool, false, src_blk, S_init, stream);
}

lkv_status lkv_init_single_bf16(const lkv_layer* L, int32_t n_req, int32_t n_blk, const void* B_pool,
                                const int32_t* src_blk, float* S_init, void* stream) {
    return init_single(L, n_req, n_blk, B_pool, true, src_blk, S_init, stream);
}

lkv_status lkv_init_compose(const lkv_layer* L, int32_t n_req, int32_t n_blk, const float* B_pool,
                            const float* M_pool, const int32_t* blk_ids, const int32_t* blk_cu, int32_t n_ids,
                            float* S_init, void* stream) {
    return init_compose(L, n_req, n_blk, B_pool, false, M_pool, blk_ids, blk_cu, n_ids, S_init, stream);
}

lkv_status lkv_init_compose_bf16(const lkv_layer* L, int32_t n_req, int32_t n_blk, const void* B_pool,
                                 const float* M_pool, const int32_t* blk_ids, const int32_t* blk_cu, int32_t n_ids,
                                 float* S_init, void* stream) {
    return init_compose(L, n_req, n_blk, B_pool, true, M_pool, blk_ids, blk_cu, n_ids, S_init, stream);
}

lkv_status lkv_round_bf16(const float* src, void* dst, int64_t n, void* stream) {
    if (n < 0) return LKV_E_SHAPE;
    if (n == 0) return LKV_OK;
    if (!src || !dst) return LKV_E_NULL;
    if (!aligned16(src) || !aligned16(dst)) return LKV_E_ALIGN;
    return hip_status(launch_round_bf16(src, dst, n, (hipStream_t)stream));
}

lkv_status lkv_stage_rows(void* dst, const void* src, const int32_t* rows, int32_t n_rows, int64_t row_bytes,
                          void* stream) {
    if (n_rows < 0 || row_bytes < 0) return LKV_E_SHAPE;
    if (n_rows == 0 || row_bytes == 0) return LKV_OK;
    if (!dst || !src || !rows) return LKV_E_NULL;
    for (int32_t i = 0; i < n_rows; ++i)
        if (rows[i] < 0) return LKV_E_SHAPE;
    return hip_status(stage_rows(dst, src, rows, n_rows, row_bytes, (hipStream_t)stream));
}

lkv_status lkv_gdn_chunk_scan(const lkv_layer* L, const lkv_tokens* T, float scale, const float* S_init,
                              void* o, float* S_final, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (L->family != LKV_GDN) return LKV_E_SHAPE;
    return chunk_scan(L, T, scale, S_init, o, S_final, stream);
}

lkv_status lkv_ssd_chunk_scan(const lkv_layer* L, const lkv_tokens* T, const float* S_init, void* y,
                              float* S_final, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (L->family != LKV_SSD) return LKV_E_SHAPE;
    return chunk_scan(L, T, 1.f, S_init, y, S_final, stream);
}

lkv_status lkv_gdn_decode(const lkv_layer* L, int32_t n_req, const void* q, const void* k, const void* v,
                          const void* g, const void* beta, float scale, float* S, void* o, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (L->family != LKV_GDN) return LKV_E_SHAPE;
    return decode(L, n_req, q, k, v, g, beta, nullptr, scale, S, o, stream);
}

lkv_status lkv_ssd_decode(const lkv_layer* L, int32_t n_req, const void* C, const void* B, const void* x,
                          const float* dt, const float* A, float* S, void* y, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (L->family != LKV_SSD) return LKV_E_SHAPE;
    if (n_req > 0 && !A) return LKV_E_NULL;
    return decode(L, n_req, C, B, x, dt, nullptr, A, 1.f, S, y, stream);
}

lkv_status lkv_gather_selected(const lkv_layer* L, const lkv_tokens* ctx, const int32_t* pos,
                               const int32_t* sel_cu, int64_t n_sel, void* q, void* k, void* v, void* g,
                               void* beta, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (!ctx) return LKV_E_NULL;
    if (n_sel < 0 || ctx->n_seq < 0 || ctx->n_tok < 0) return LKV_E_SHAPE;
    if (n_sel == 0) return LKV_OK;
    if (n_sel >= (INT64_C(1) << 31)) return LKV_E_SHAPE;
    if (!pos || !sel_cu || !ctx->cu) return LKV_E_NULL;
    const int io = L->io_dtype == LKV_BF16 ? 2 : 4;
    const int gate = (L->family == LKV_GDN && L->gate_dtype == LKV_BF16) ? 2 : 4;
    GatherArgs a = {};
    a.ctx_cu = ctx->cu;
    a.ctx_tok = ctx->n_tok;
    a.pos = pos;
    a.sel_cu = sel_cu;
    a.n_sel = n_sel;
    a.n_req = ctx->n_seq;
    const void* src[GATHER_ARRAYS] = {ctx->q, ctx->k, ctx->v, ctx->g, ctx->beta};
    void* dst[GATHER_ARRAYS] = {q, k, v, g, L->family == LKV_GDN ? beta : nullptr};
    const int64_t rb[GATHER_ARRAYS] = {(int64_t)L->h_qk * L->dk * io, (int64_t)L->h_qk * L->dk * io,
                                       (int64_t)L->h_v * L->dv * io, (int64_t)L->h_v * gate,
                                       (int64_t)L->h_v * gate};
    const int eb[GATHER_ARRAYS] = {io, io, io, gate, gate};
    bool any = false;
    for (int i = 0; i < GATHER_ARRAYS; ++i) {
        if (!dst[i]) continue;
        if (!src[i]) return LKV_E_NULL;
        if (!aligned16(src[i]) || !aligned16(dst[i])) return LKV_E_ALIGN;
        if (rb[i] >= (INT64_C(1) << 30)) return LKV_E_SHAPE;
        a.src[i] = src[i];
        a.dst[i] = dst[i];
        a.row_bytes[i] = (int32_t)rb[i];
        a.elem_bytes[i] = eb[i];
        any = true;
    }
    if (!any) return LKV_OK;
    if (ctx->n_seq == 0) return LKV_E_SHAPE;
    return hip_status(launch_gather(a, (hipStream_t)stream));
}

lkv_status lkv_state_rel_error(const float* S, const float* S_ref, int32_t n_slices, int64_t slice_elems,
                               int32_t group, double* sq, double* rel, double* rel_group, void* stream) {
    if (n_slices < 0 || slice_elems < 0) return LKV_E_SHAPE;
    if (n_slices == 0) return LKV_OK;
    if (!S || !S_ref || !sq || !rel) return LKV_E_NULL;
    if (slice_elems % 4 != 0) return LKV_E_SHAPE;
    if (rel_group && (group < 1 || n_slices % group != 0)) return LKV_E_SHAPE;
    if (!aligned16(S) || !aligned16(S_ref)) return LKV_E_ALIGN;
    return hip_status(launch_rel_error(S, S_ref, n_slices, slice_elems, group, sq, rel, rel_group,
                                       (hipStream_t)stream));
}

lkv_status lkv_chunk_scan_from_pool(const lkv_layer* L, const lkv_tokens* T, float scale, const void* B_pool,
                                    int32_t pool_dtype, int32_t n_blk, const int32_t* src_blk, void* out,
                                    float* S_final, void* stream) {
    lkv_status s = check_layer(L);
    if (s != LKV_OK) return s;
    if (!T) return LKV_E_NULL;
    if (n_blk < 0) return LKV_E_SHAPE;
    if (pool_dtype != LKV_F32 && pool_dtype != LKV_BF16) return LKV_E_DTYPE;
    if (T->n_seq > 0 && !src_blk) return LKV_E_NULL;
    if (n_blk > 0 && !B_pool) return LKV_E_NULL;
    if (B_pool && !aligned16(B_pool)) return LKV_E_ALIGN;
    // with n_blk = 0 every id is -1 (zero state) or invalid (NaN): the pool is never read
    return chunk_scan(L, T, L->family == LKV_GDN ? scale : 1.f, reinterpret_cast<const float*>(B_pool), out,
                      S_final, stream, src_blk, n_blk, pool_dtype == LKV_BF16);
}

lkv_status lkv_chunk_scan_sp_workspace(const lkv_layer* L, int32_t n_req, int32_t pieces, size_t* bytes) {
    if (!bytes) return LKV_E_NULL;
    lkv_status s = sp_check(L, n_req, pieces);
    if (s != LKV_OK) return s;
    *bytes = sp_layout(L, n_req, pieces).total;
    return LKV_OK;
}

lkv_status lkv_chunk_scan_sp(const lkv_layer* L, const lkv_tokens* T, float scale, const float* S_init, void* out,
                             float* S_final, int32_t pieces, void* ws, size_t ws_bytes, void* stream) {
    return chunk_scan_sp(L, T, scale, S_init, out, S_final, pieces, reinterpret_cast<char*>(ws), ws_bytes, stream);
}

lkv_status lkv_chunk_scan_sp_noalloc(const lkv_layer* L, const lkv_tokens* T, float scale, const float* S_init,
                                     void* out, float* S_final, int32_t pieces, void* stream) {
    if (!T) return LKV_E_NULL;
    lkv_status s = sp_check(L, T->n_seq, pieces);
    if (s != LKV_OK) return s;
    if (sp_layout(L, T->n_seq, pieces).total > kScratchBytes) return LKV_E_WORKSPACE;
    char* ws = nullptr;
    s = scratch_for_current_device(&ws);
    if (s != LKV_OK) return s;
    return chunk_scan_sp(L, T, scale, S_init, out, S_final, pieces, ws, kScratchBytes, stream);
}

}  // extern "C"
