// spire_abi.hip -- host implementation of the C ABI in include/spire.h.
//
// Validates arguments, lays out the caller's workspace, picks the kernel
// family (matrix-core for bf16/fp8 K/V with head_dim 128, generic otherwise)
// and enqueues plan -> partial attention -> combine on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include <cmath>

#include "spire_internal.h"

using namespace spire;

namespace {

thread_local char g_err[512] = "";

spire_status fail(spire_status s, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return s;
}

// ---- device properties ------------------------------------------------------
constexpr int kMaxDevices = 64;
int g_cus[kMaxDevices] = {0};
std::mutex g_dev_mu;

int device_cus(int *cus_out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return -1;
    std::lock_guard<std::mutex> lock(g_dev_mu);
    if (g_cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            return -1;
        g_cus[dev] = n;
    }
    *cus_out = g_cus[dev];
    return 0;
}

// ---- library-owned scratch of the entry point that allocates nothing ---------
// spire_verify_attn_noalloc runs the kernels of spire_verify_attn with this
// array as their workspace.  Each device holds its own copy from the library's
// load until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory: only the address hipGetSymbolAddress returns
// for the current device may reach a kernel.
constexpr size_t kScratchBytes = (size_t)80 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];
void *g_scratch[kMaxDevices] = {nullptr};  // device address of `scratch`, set once per device

spire_status scratch_address(void **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return fail(SPIRE_ERR_HIP, "cannot query the current HIP device");
    std::lock_guard<std::mutex> lock(g_dev_mu);
    if (g_scratch[dev] == nullptr) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || ptr == nullptr)
            return fail(SPIRE_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return SPIRE_OK;
}

// ---- workspace layout -------------------------------------------------------
struct Layout {
    size_t nkeys, prefix, wstart, part_lse, part_o, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Layout layout(int64_t B, int64_t rows, int64_t D, int64_t workers) {
    Layout L;
    size_t off = 0;
    L.nkeys = off; off = align256(off + 4 * (size_t)B);
    L.prefix = off; off = align256(off + 4 * (size_t)(B + 1));
    L.wstart = off; off = align256(off + 8 * (size_t)workers);
    L.part_lse = off; off = align256(off + 4 * (size_t)(2 * workers * rows));
    L.part_o = off; off = align256(off + 4 * (size_t)(2 * workers * rows * D));
    L.total = off;
    return L;
}

// One wave per SIMD: measured faster than two for the register-staged kernel
// (two waves halve the tiles each keeps in flight).
int mfma_workers(int cus) { return cus * kMfmaWavesPerWG; }
int generic_workers(int cus) { return cus * kMaxWorkersPerCU; }

size_t workspace_bytes_for(int B, int R, int D) {
    int cus = 0;
    if (device_cus(&cus) != 0) return 0;
    // the largest launch of any kernel that may serve R rows, either K/V dtype
    const int nb = (R + 15) / 16;
    int w = 0;
    for (bool fp8 : {false, true}) {
        w = std::max(w, mfma_workers(cus));
        w = std::max(w, staged_workers(cus, nb, fp8));
    }
    const Layout a = layout(B, R, D, w);
    const Layout b = layout(B, kGenericRowBlock, D, generic_workers(cus));
    return a.total > b.total ? a.total : b.total;
}

// ---- per-call options: kernel family and launch events ----------------------------
// Kernel ids of the recorded launches (include/spire.h).
enum { KID_PLAN = 0, KID_VERIFY = 1, KID_DRAFT = 2, KID_COMBINE = 3, KID_TOKEN_WEIGHTS = 4,
       KID_TOKEN_SELECT = 5, KID_TAIL_CHECK = 11, KID_BLOCK_WEIGHTS = 12, KID_BLOCK_SELECT = 13 };

// Records the caller's events around each launch of one call, in launch order.
struct Recorder {
    const spire_launch_opts *o;
    int n = 0;
    explicit Recorder(const spire_launch_opts *opts) : o(opts) {}
    template <class F>
    hipError_t run(int id, hipStream_t st, F &&launch) {
        const bool rec = o != nullptr && o->events != nullptr && n < o->max_launches;
        hipError_t e = hipSuccess;
        if (rec && (e = hipEventRecord(o->events[2 * n], st)) != hipSuccess) return e;
        if ((e = launch()) != hipSuccess) return e;
        if (rec) {
            if ((e = hipEventRecord(o->events[2 * n + 1], st)) != hipSuccess) return e;
            if (o->kernel_ids != nullptr) o->kernel_ids[n] = id;
        }
        ++n;
        return hipSuccess;
    }
    hipError_t run(int id, hipStream_t st, hipError_t (*fn)(const Problem &, const Plan &, hipStream_t),
                   const Problem &p, const Plan &pl) {
        return run(id, st, [&] { return fn(p, pl, st); });
    }
    ~Recorder() {
        if (o != nullptr && o->n_launches != nullptr) *o->n_launches = n;
    }
};

spire_status check_opts(const spire_launch_opts *o) {
    if (o == nullptr) return SPIRE_OK;
    if (o->kernel < 0 || o->kernel > 3) return fail(SPIRE_ERR_INVALID_ARG, "opts->kernel must be 0..3 (got %d)", o->kernel);
    if (o->max_launches < 0) return fail(SPIRE_ERR_INVALID_ARG, "opts->max_launches must be >= 0");
    if (o->max_launches > 0 && o->events == nullptr)
        return fail(SPIRE_ERR_INVALID_ARG, "opts->events is NULL with max_launches > 0");
    if (o->reserved != 0) return fail(SPIRE_ERR_INVALID_ARG, "opts->reserved must be 0");
    return SPIRE_OK;
}

// ---- argument checks --------------------------------------------------------
bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int elem_size(int dt) {
    switch (dt) {
    case SPIRE_F32: return 4;
    case SPIRE_BF16: return 2;
    case SPIRE_FP8_E4M3FN: return 1;
    default: return 0;
    }
}

spire_status check_kv(const spire_kv *kv, const char *name, int D, int Hkv, bool allow_paged,
                      bool read = true) {
    if (kv == nullptr) return fail(SPIRE_ERR_INVALID_ARG, "%s: descriptor is NULL", name);
    if (read && (kv->k == nullptr || kv->v == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "%s: k or v is NULL", name);
    const int es = elem_size(kv->dtype);
    if (es == 0) return fail(SPIRE_ERR_INVALID_ARG, "%s: unknown dtype %d", name, kv->dtype);
    if (kv->reserved != 0) return fail(SPIRE_ERR_INVALID_ARG, "%s: reserved field must be 0", name);
    if (kv->s_blk < 0 || kv->s_head < 0 || kv->s_tok < 0)
        return fail(SPIRE_ERR_INVALID_ARG, "%s: negative stride", name);
    if (read && kv->dtype == SPIRE_FP8_E4M3FN && (kv->k_scale == nullptr || kv->v_scale == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "%s: fp8 storage needs k_scale and v_scale", name);
    if (kv->page_size < 0) return fail(SPIRE_ERR_INVALID_ARG, "%s: negative page_size", name);
    if (kv->page_size > 0) {
        if (!allow_paged) return fail(SPIRE_ERR_UNSUPPORTED, "%s: paged storage not supported here", name);
        if (kv->block_table == nullptr || kv->max_blocks <= 0 || kv->num_blocks <= 0)
            return fail(SPIRE_ERR_INVALID_ARG, "%s: paged view needs block_table, max_blocks > 0, num_blocks > 0", name);
    } else {
        if (kv->capacity < 0) return fail(SPIRE_ERR_INVALID_ARG, "%s: negative capacity", name);
    }
    (void)D; (void)Hkv;
    return SPIRE_OK;
}

KvDev to_dev(const spire_kv *kv) {
    KvDev d;
    d.k = static_cast<const uint8_t *>(kv->k);
    d.v = static_cast<const uint8_t *>(kv->v);
    d.block_table = kv->block_table;
    d.k_scale = kv->k_scale;
    d.v_scale = kv->v_scale;
    d.s_blk = kv->s_blk;
    d.s_head = kv->s_head;
    d.s_tok = kv->s_tok;
    d.elem = elem_size(kv->dtype);
    d.page_size = kv->page_size;
    d.max_blocks = kv->max_blocks;
    d.num_blocks = kv->num_blocks;
    d.capacity = kv->capacity;
    return d;
}

bool rows_aligned(const spire_kv *kv) {
    const int es = elem_size(kv->dtype);
    return aligned16(kv->k) && aligned16(kv->v) && (kv->s_blk * es) % 16 == 0 &&
           (kv->s_head * es) % 16 == 0 && (kv->s_tok * es) % 16 == 0;
}

spire_status common_checks(const void *q, int q_dtype, int B, int Hq, int Hkv, int D, int k,
                           const void *out, int out_dtype, const void *workspace) {
    if (B < 0) return fail(SPIRE_ERR_INVALID_ARG, "B must be >= 0 (got %d)", B);
    if (Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0)
        return fail(SPIRE_ERR_INVALID_ARG, "need Hkv >= 1 and Hq %% Hkv == 0 (Hq=%d, Hkv=%d)", Hq, Hkv);
    if (D != 64 && D != 128) return fail(SPIRE_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", D);
    if (k < 0 || k > 15) return fail(SPIRE_ERR_UNSUPPORTED, "k must be in [0, 15] (got %d)", k);
    if ((int64_t)(k + 1) * (Hq / Hkv) > kMaxRows)
        return fail(SPIRE_ERR_UNSUPPORTED, "(k+1)*Hq/Hkv = %d exceeds %d", (k + 1) * (Hq / Hkv), kMaxRows);
    if (q_dtype != SPIRE_F32 && q_dtype != SPIRE_BF16)
        return fail(SPIRE_ERR_UNSUPPORTED, "q_dtype must be F32 or BF16");
    if (out_dtype != SPIRE_F32 && out_dtype != SPIRE_BF16)
        return fail(SPIRE_ERR_UNSUPPORTED, "out_dtype must be F32 or BF16");
    if (B > 0 && (q == nullptr || out == nullptr)) return fail(SPIRE_ERR_INVALID_ARG, "q or out is NULL");
    if (B > 0 && workspace == nullptr) return fail(SPIRE_ERR_WORKSPACE, "workspace is NULL");
    if (B > kPlanMaxB) return fail(SPIRE_ERR_UNSUPPORTED, "B must be <= %d (got %d)", kPlanMaxB, B);
    if (!aligned16(q) || !aligned16(out)) return fail(SPIRE_ERR_INVALID_ARG, "q and out must be 16-byte aligned");
    if (((uintptr_t)workspace & 255u) != 0) return fail(SPIRE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    return SPIRE_OK;
}

// Kernel family for a matrix-core eligible request: LDS-staged for more than
// 32 rows (deep stage ring; the row blocks on two waves, or all five fp8
// blocks of 72-80 rows on one; up to 8 blocks, 128 rows), register-staged
// otherwise; the caller's kernel choice can ask for the LDS-staged one.
bool use_staged(const Problem &p, int kernel) {
    const int nb = (p.R + 15) / 16;
    if (nb > 2) return true;  // the register-staged kernel holds at most 32 rows
    if (kernel == 3) return p.kv_dtype == SPIRE_FP8_E4M3FN;
    return false;  // measured: up to 32 rows the register-staged kernel is faster
}

// Waves per segment for a draft step with whole segments per workgroup, or 0
// for the stream-K partition: 4 or 2 waves per segment when that fills at
// least 15/16 of the device's waves without exceeding them (a draft segment
// never exceeds S + W keys, so equal shares of segments stay balanced).
// Kernel choice 2 keeps the stream-K partition.
int draft_coop_waves(const Problem &p, int cus, int kernel) {
    if (!p.draft || kernel == 2) return 0;
    const int64_t segs = (int64_t)p.B * p.Hkv, waves = mfma_workers(cus);
    if (segs <= 0) return 0;
    for (int g = kMfmaWavesPerWG; g >= 2; g /= 2)
        if (segs * g <= waves && segs * g * 16 >= waves * 15) return g;
    return 0;
}

spire_status run(Problem &p, bool use_mfma, void *workspace, size_t ws_bytes, hipStream_t stream,
                 int partial_id, const spire_launch_opts *opts, bool lib_scratch = false) {
    int cus = 0;
    if (device_cus(&cus) != 0) return fail(SPIRE_ERR_HIP, "cannot query the current HIP device");
    const int kernel = opts != nullptr ? opts->kernel : 0;
    Recorder rec(opts);
    const bool mf = use_mfma && kernel != 1;
    const bool staged = mf && use_staged(p, kernel);
    const int nb = (p.R + 15) / 16;
    Plan pl;
    pl.tile = mf ? kMfmaTile : kGenericTile;
    const int nrb = mf ? 1 : (p.R + kGenericRowBlock - 1) / kGenericRowBlock;
    pl.units = p.Hkv * nrb;
    pl.rows = mf ? p.R : kGenericRowBlock;
    pl.workers = !mf ? generic_workers(cus)
                     : (staged ? staged_workers(cus, nb, p.kv_dtype == SPIRE_FP8_E4M3FN)
                               : mfma_workers(cus));
    // phantom positions per segment (spire_internal.h): on the matrix-core
    // kernels a worker's time grew by about as much per segment it covered as
    // streaming 35-40 KB of keys takes (queries, output rows, address set-up,
    // pipeline refill); without this, workers covering many short sequences
    // finished last
    const int64_t tile_bytes = 2LL * kMfmaTile * p.D * p.kv.elem;
    pl.seg_cost = mf ? (int)((40960 + tile_bytes / 2) / tile_bytes) : 0;
    if (pl.workers > kCombineMaxWorkers)
        return fail(SPIRE_ERR_UNSUPPORTED, "%d workers exceed the combine's limit of %d", pl.workers,
                    kCombineMaxWorkers);
    const Layout L = layout(p.B, pl.rows, p.D, pl.workers);
    if (ws_bytes < L.total && lib_scratch)
        return fail(SPIRE_ERR_UNSUPPORTED,
                    "this call needs %zu bytes of scratch; the no-allocation entry point holds %zu per device "
                    "(use spire_verify_attn with a workspace)", L.total, ws_bytes);
    if (ws_bytes < L.total)
        return fail(SPIRE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, L.total);
    char *ws = static_cast<char *>(workspace);
    pl.nkeys = reinterpret_cast<int32_t *>(ws + L.nkeys);
    pl.prefix = reinterpret_cast<int32_t *>(ws + L.prefix);
    pl.wstart = reinterpret_cast<int32_t *>(ws + L.wstart);
    pl.part_lse = reinterpret_cast<float *>(ws + L.part_lse);
    pl.part_o = reinterpret_cast<float *>(ws + L.part_o);

    hipError_t e = hipSuccess;
    if (const int g = (mf && !staged) ? draft_coop_waves(p, cus, kernel) : 0) {
        e = rec.run(partial_id, stream, [&] { return launch_mfma_draft_coop(p, nb, g, stream); });
        if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "attention launch: %s", hipGetErrorString(e));
        return SPIRE_OK;
    }
    // the register-staged kernel computes the partition itself; the others
    // read it from the plan kernel's output
    if (!mf || staged) {
        e = rec.run(KID_PLAN, stream, launch_plan, p, pl);
        if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "plan launch: %s", hipGetErrorString(e));
    }
    if (staged) {
        auto fn = [](const Problem &pp, const Plan &pp2, hipStream_t s) {
            return launch_staged_partial(pp, pp2, (pp.R + 15) / 16, s);
        };
        e = rec.run(partial_id, stream, fn, p, pl);
    } else if (mf) {
        auto fn = [](const Problem &pp, const Plan &pp2, hipStream_t s) {
            return launch_mfma_partial(pp, pp2, (pp.R + 15) / 16, s);
        };
        e = rec.run(partial_id, stream, fn, p, pl);
    } else {
        e = rec.run(partial_id, stream, launch_generic_partial, p, pl);
    }
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "attention launch: %s", hipGetErrorString(e));
    e = rec.run(KID_COMBINE, stream, launch_combine, p, pl);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "combine launch: %s", hipGetErrorString(e));
    // the matrix-core kernels multiply the values of keys a row masks by zero:
    // segments with a non-finite value among keys [n - k, n) are redone exactly
    if (mf && !p.draft && p.k > 0) {
        e = rec.run(KID_TAIL_CHECK, stream, launch_tail_fix, p, pl);
        if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "tail check launch: %s", hipGetErrorString(e));
    }
    return SPIRE_OK;
}

}  // namespace

extern "C" {

int32_t spire_version(void) { return SPIRE_VERSION; }

const char *spire_status_string(int32_t s) {
    switch (s) {
    case SPIRE_OK: return "SPIRE_OK";
    case SPIRE_ERR_INVALID_ARG: return "SPIRE_ERR_INVALID_ARG";
    case SPIRE_ERR_UNSUPPORTED: return "SPIRE_ERR_UNSUPPORTED";
    case SPIRE_ERR_WORKSPACE: return "SPIRE_ERR_WORKSPACE";
    case SPIRE_ERR_HIP: return "SPIRE_ERR_HIP";
    default: return "SPIRE_ERR_UNKNOWN";
    }
}

const char *spire_last_error(void) { return g_err; }

size_t spire_verify_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t D, int32_t k) {
    if (B < 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || D <= 0 || k < 0) return 0;
    return workspace_bytes_for(B, (k + 1) * (Hq / Hkv), D);
}

size_t spire_draft_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t D) {
    if (B < 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || D <= 0) return 0;
    return workspace_bytes_for(B, Hq / Hkv, D);
}

// The kernels take row maxima of raw scores, which needs a positive scale.
static spire_status check_scale(float sm_scale) {
    if (!(sm_scale > 0.f) || !std::isfinite(sm_scale))
        return fail(SPIRE_ERR_INVALID_ARG, "sm_scale must be finite and > 0 (got %g)", (double)sm_scale);
    return SPIRE_OK;
}

spire_status spire_verify_attn(const void *q, int32_t q_dtype, const spire_kv *kv,
                               const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                               int32_t D, int32_t k, float sm_scale, void *out,
                               int32_t out_dtype, float *lse, void *workspace,
                               size_t workspace_bytes, hipStream_t stream) {
    return spire_verify_attn_ex(q, q_dtype, kv, kv_lens, B, Hq, Hkv, D, k, sm_scale, out, out_dtype, lse,
                                workspace, workspace_bytes, stream, nullptr);
}

static spire_status verify_impl(const void *q, int32_t q_dtype, const spire_kv *kv,
                                const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                int32_t D, int32_t k, float sm_scale, void *out,
                                int32_t out_dtype, float *lse, void *workspace,
                                size_t workspace_bytes, hipStream_t stream,
                                const spire_launch_opts *opts, bool lib_scratch);

spire_status spire_verify_attn_ex(const void *q, int32_t q_dtype, const spire_kv *kv,
                                  const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                  int32_t D, int32_t k, float sm_scale, void *out,
                                  int32_t out_dtype, float *lse, void *workspace,
                                  size_t workspace_bytes, hipStream_t stream,
                                  const spire_launch_opts *opts) {
    g_err[0] = '\0';
    return verify_impl(q, q_dtype, kv, kv_lens, B, Hq, Hkv, D, k, sm_scale, out, out_dtype, lse, workspace,
                       workspace_bytes, stream, opts, false);
}

spire_status spire_verify_attn_noalloc(const void *q, int32_t q_dtype, const spire_kv *kv,
                                       const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                       int32_t D, int32_t k, float sm_scale, void *out,
                                       int32_t out_dtype, float *lse, hipStream_t stream) {
    g_err[0] = '\0';
    void *ws = nullptr;
    if (B > 0) {
        const spire_status s = scratch_address(&ws);
        if (s != SPIRE_OK) return s;
    }
    return verify_impl(q, q_dtype, kv, kv_lens, B, Hq, Hkv, D, k, sm_scale, out, out_dtype, lse, ws,
                       B > 0 ? kScratchBytes : 0, stream, nullptr, true);
}

static spire_status verify_impl(const void *q, int32_t q_dtype, const spire_kv *kv,
                                const int32_t *kv_lens, int32_t B, int32_t Hq, int32_t Hkv,
                                int32_t D, int32_t k, float sm_scale, void *out,
                                int32_t out_dtype, float *lse, void *workspace,
                                size_t workspace_bytes, hipStream_t stream,
                                const spire_launch_opts *opts, bool lib_scratch) {
    if (opts != nullptr && opts->n_launches != nullptr) *opts->n_launches = 0;
    spire_status s = check_opts(opts);
    if (s != SPIRE_OK) return s;
    s = common_checks(q, q_dtype, B, Hq, Hkv, D, k, out, out_dtype, workspace);
    if (s != SPIRE_OK) return s;
    s = check_scale(sm_scale);
    if (s != SPIRE_OK) return s;
    s = check_kv(kv, "kv", D, Hkv, true);
    if (s != SPIRE_OK) return s;
    if (B > 0 && kv_lens == nullptr) return fail(SPIRE_ERR_INVALID_ARG, "kv_lens is NULL");
    if (kv->page_size == 0 && kv->capacity <= 0 && B > 0)
        return fail(SPIRE_ERR_INVALID_ARG, "contiguous kv needs capacity > 0");
    if (B == 0) return SPIRE_OK;

    Problem p;
    memset(&p, 0, sizeof p);
    p.draft = 0;
    p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.D = D; p.k = k;
    p.g = Hq / Hkv;
    p.R = (k + 1) * p.g;
    p.sm_scale_log2 = sm_scale * 1.4426950408889634f;
    p.q = static_cast<const uint8_t *>(q);
    p.q_dtype = q_dtype;
    p.kv_dtype = kv->dtype;
    p.lens = kv_lens;
    p.kv = to_dev(kv);
    p.out = out;
    p.out_dtype = out_dtype;
    p.lse = lse;

    // paged: 16-key groups never straddle a page, and the matrix-core kernels
    // form page offsets with 32-bit products
    const int es = elem_size(kv->dtype);
    // paged: 16-key groups never straddle a page, and the matrix-core kernels
    // form page offsets with 32-bit products; both layouts: 16 key rows span
    // under 2^31 bytes (32-bit lane offsets of the loads)
    const bool layout_ok =
        (uint64_t)kv->s_tok * es * 16 < (1ull << 31) &&
        (kv->page_size > 0
             ? (kv->page_size % 16 == 0 && (uint64_t)kv->s_blk * es < (1ull << 32) &&
                (uint64_t)kv->page_size * kv->s_tok * es < (1ull << 31))
             : (kv->capacity >= 1));
    const bool mfma = (kv->dtype == SPIRE_BF16 || kv->dtype == SPIRE_FP8_E4M3FN) &&
                      q_dtype == SPIRE_BF16 && D == 128 && p.R <= kMaxRows && layout_ok && rows_aligned(kv);
    return run(p, mfma, workspace, workspace_bytes, stream, KID_VERIFY, opts, lib_scratch);
}

spire_status spire_draft_sparse_attn(const void *q, int32_t q_dtype, const spire_kv *sink,
                                     const spire_kv *ring, const int32_t *seq_lens,
                                     const int32_t *ring_offset, int32_t B, int32_t Hq,
                                     int32_t Hkv, int32_t D, int32_t S, int32_t W, float sm_scale,
                                     void *out, int32_t out_dtype, float *lse, void *workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
    return spire_draft_sparse_attn_ex(q, q_dtype, sink, ring, seq_lens, ring_offset, B, Hq, Hkv, D, S, W, sm_scale,
                                      out, out_dtype, lse, workspace, workspace_bytes, stream, nullptr);
}

spire_status spire_draft_sparse_attn_ex(const void *q, int32_t q_dtype, const spire_kv *sink,
                                        const spire_kv *ring, const int32_t *seq_lens,
                                        const int32_t *ring_offset, int32_t B, int32_t Hq,
                                        int32_t Hkv, int32_t D, int32_t S, int32_t W, float sm_scale,
                                        void *out, int32_t out_dtype, float *lse, void *workspace,
                                        size_t workspace_bytes, hipStream_t stream,
                                        const spire_launch_opts *opts) {
    g_err[0] = '\0';
    if (opts != nullptr && opts->n_launches != nullptr) *opts->n_launches = 0;
    spire_status s = check_opts(opts);
    if (s != SPIRE_OK) return s;
    s = common_checks(q, q_dtype, B, Hq, Hkv, D, 0, out, out_dtype, workspace);
    if (s != SPIRE_OK) return s;
    s = check_scale(sm_scale);
    if (s != SPIRE_OK) return s;
    if (S < 0 || W < 0 || (int64_t)S + W < 1)
        return fail(SPIRE_ERR_INVALID_ARG, "need S >= 0, W >= 0, S + W >= 1 (S=%d, W=%d)", S, W);
    s = check_kv(sink, "sink", D, Hkv, false, S > 0);
    if (s != SPIRE_OK) return s;
    s = check_kv(ring, "ring", D, Hkv, false, W > 0);
    if (s != SPIRE_OK) return s;
    if (sink->dtype != ring->dtype) return fail(SPIRE_ERR_INVALID_ARG, "sink and ring dtypes differ");
    if (sink->capacity < S) return fail(SPIRE_ERR_INVALID_ARG, "sink capacity %d < S = %d", sink->capacity, S);
    if (ring->capacity < W) return fail(SPIRE_ERR_INVALID_ARG, "ring capacity %d < W = %d", ring->capacity, W);
    if (B > 0 && (seq_lens == nullptr || ring_offset == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "seq_lens or ring_offset is NULL");
    if (B == 0) return SPIRE_OK;

    Problem p;
    memset(&p, 0, sizeof p);
    p.draft = 1;
    p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.D = D; p.k = 0;
    p.g = Hq / Hkv;
    p.R = p.g;
    p.S = S; p.W = W;
    p.sm_scale_log2 = sm_scale * 1.4426950408889634f;
    p.q = static_cast<const uint8_t *>(q);
    p.q_dtype = q_dtype;
    p.kv_dtype = ring->dtype;
    p.lens = seq_lens;
    p.ring_offset = ring_offset;
    p.kv = to_dev(ring);
    p.sink = to_dev(sink);
    p.out = out;
    p.out_dtype = out_dtype;
    p.lse = lse;

    const bool same_scales = ring->dtype != SPIRE_FP8_E4M3FN ||
                             (ring->k_scale == sink->k_scale && ring->v_scale == sink->v_scale);
    // 16 ring rows span under 2^31 bytes (32-bit lane offsets of the loads)
    const bool mfma = (ring->dtype == SPIRE_BF16 || ring->dtype == SPIRE_FP8_E4M3FN) &&
                      q_dtype == SPIRE_BF16 && D == 128 && p.R <= kMaxRows && same_scales &&
                      (uint64_t)ring->s_tok * elem_size(ring->dtype) * 16 < (1ull << 31) &&
                      rows_aligned(ring) && rows_aligned(sink);
    return run(p, mfma, workspace, workspace_bytes, stream, KID_DRAFT, opts);
}

// ---- token verification -------------------------------------------------------

static int token_pieces(int32_t V) { return (V + kTokenPiece - 1) / kTokenPiece; }

size_t spire_token_verify_workspace_size(int32_t B, int32_t k, int32_t V) {
    if (B < 0 || k < 0 || k > kTokenMaxK || V < 1 || V > kTokenMaxV) return 0;
    return align256((size_t)B * token_pieces(V) * sizeof(uint64_t)) + align256(4 * (size_t)B + 1);
}

spire_status spire_token_verify(const float *p_target, const float *q_draft,
                                const int32_t *draft_tokens, const float *u_accept,
                                const float *u_sample, int32_t B, int32_t k, int32_t V,
                                int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                size_t workspace_bytes, hipStream_t stream) {
    return spire_token_verify_ex(p_target, q_draft, draft_tokens, u_accept, u_sample, B, k, V, n_accepted,
                                 out_tokens, workspace, workspace_bytes, stream, nullptr);
}

spire_status spire_token_verify_ex(const float *p_target, const float *q_draft,
                                   const int32_t *draft_tokens, const float *u_accept,
                                   const float *u_sample, int32_t B, int32_t k, int32_t V,
                                   int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream,
                                   const spire_launch_opts *opts) {
    g_err[0] = '\0';
    if (opts != nullptr && opts->n_launches != nullptr) *opts->n_launches = 0;
    if (check_opts(opts) != SPIRE_OK) return SPIRE_ERR_INVALID_ARG;
    if (B < 0 || B > 65535) return fail(SPIRE_ERR_UNSUPPORTED, "B must be in [0, 65535] (got %d)", B);
    if (k < 0 || k > kTokenMaxK) return fail(SPIRE_ERR_UNSUPPORTED, "k must be in [0, %d] (got %d)", kTokenMaxK, k);
    if (V < 1 || V > kTokenMaxV) return fail(SPIRE_ERR_UNSUPPORTED, "V must be in [1, %d] (got %d)", kTokenMaxV, V);
    if (B == 0) return SPIRE_OK;
    if (p_target == nullptr || u_sample == nullptr || n_accepted == nullptr || out_tokens == nullptr)
        return fail(SPIRE_ERR_INVALID_ARG, "p_target, u_sample, n_accepted or out_tokens is NULL");
    if (k > 0 && (q_draft == nullptr || draft_tokens == nullptr || u_accept == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "q_draft, draft_tokens or u_accept is NULL with k > 0");
    const void *ptrs[] = {p_target, q_draft, draft_tokens, u_accept, u_sample, n_accepted, out_tokens};
    for (const void *ptr : ptrs)
        if (((uintptr_t)ptr & 3u) != 0) return fail(SPIRE_ERR_INVALID_ARG, "arrays must be 4-byte aligned");
    const size_t need = spire_token_verify_workspace_size(B, k, V);
    if (workspace == nullptr) return fail(SPIRE_ERR_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(SPIRE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(SPIRE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    TokenProblem t;
    t.p = p_target;
    t.q = q_draft;
    t.draft = draft_tokens;
    t.u_accept = u_accept;
    t.u_sample = u_sample;
    t.B = B;
    t.k = k;
    t.V = V;
    t.npieces = token_pieces(V);
    t.n_accepted = n_accepted;
    t.out_tokens = out_tokens;
    t.piece_sum = static_cast<uint64_t *>(workspace);
    t.nacc = reinterpret_cast<int32_t *>(static_cast<char *>(workspace) +
                                         align256((size_t)B * t.npieces * sizeof(uint64_t)));
    Recorder rec(opts);
    hipError_t e = rec.run(KID_TOKEN_WEIGHTS, stream, [&] { return launch_token_weights(t, stream); });
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "token weights launch: %s", hipGetErrorString(e));
    e = rec.run(KID_TOKEN_SELECT, stream, [&] { return launch_token_select(t, stream); });
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "token select launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

// ---- block verification -------------------------------------------------------

size_t spire_block_verify_workspace_size(int32_t B, int32_t k, int32_t V) {
    if (B < 0 || k < 0 || k > kTokenMaxK || V < 1 || V > kTokenMaxV) return 0;
    return align256((size_t)B * (size_t)(k + 1) * token_pieces(V) * sizeof(uint64_t)) + 256;
}

spire_status spire_block_verify(const float *p_target, const float *q_draft,
                                const int32_t *draft_tokens, const float *u_accept,
                                const float *u_sample, int32_t B, int32_t k, int32_t V,
                                int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                size_t workspace_bytes, hipStream_t stream) {
    return spire_block_verify_ex(p_target, q_draft, draft_tokens, u_accept, u_sample, B, k, V, n_accepted,
                                 out_tokens, workspace, workspace_bytes, stream, nullptr);
}

spire_status spire_block_verify_ex(const float *p_target, const float *q_draft,
                                   const int32_t *draft_tokens, const float *u_accept,
                                   const float *u_sample, int32_t B, int32_t k, int32_t V,
                                   int32_t *n_accepted, int32_t *out_tokens, void *workspace,
                                   size_t workspace_bytes, hipStream_t stream,
                                   const spire_launch_opts *opts) {
    g_err[0] = '\0';
    if (opts != nullptr && opts->n_launches != nullptr) *opts->n_launches = 0;
    if (check_opts(opts) != SPIRE_OK) return SPIRE_ERR_INVALID_ARG;
    if (B < 0 || B > 65535) return fail(SPIRE_ERR_UNSUPPORTED, "B must be in [0, 65535] (got %d)", B);
    if (k < 0 || k > kTokenMaxK) return fail(SPIRE_ERR_UNSUPPORTED, "k must be in [0, %d] (got %d)", kTokenMaxK, k);
    if (V < 1 || V > kTokenMaxV) return fail(SPIRE_ERR_UNSUPPORTED, "V must be in [1, %d] (got %d)", kTokenMaxV, V);
    if (B == 0) return SPIRE_OK;
    if (p_target == nullptr || u_sample == nullptr || n_accepted == nullptr || out_tokens == nullptr)
        return fail(SPIRE_ERR_INVALID_ARG, "p_target, u_sample, n_accepted or out_tokens is NULL");
    if (k > 0 && (q_draft == nullptr || draft_tokens == nullptr || u_accept == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "q_draft, draft_tokens or u_accept is NULL with k > 0");
    const void *ptrs[] = {p_target, q_draft, draft_tokens, u_accept, u_sample, n_accepted, out_tokens};
    for (const void *ptr : ptrs)
        if (((uintptr_t)ptr & 3u) != 0) return fail(SPIRE_ERR_INVALID_ARG, "arrays must be 4-byte aligned");
    const size_t need = spire_block_verify_workspace_size(B, k, V);
    if (workspace == nullptr) return fail(SPIRE_ERR_WORKSPACE, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(SPIRE_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(SPIRE_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    TokenProblem t;
    t.p = p_target;
    t.q = q_draft;
    t.draft = draft_tokens;
    t.u_accept = u_accept;
    t.u_sample = u_sample;
    t.B = B;
    t.k = k;
    t.V = V;
    t.npieces = token_pieces(V);
    t.n_accepted = n_accepted;
    t.out_tokens = out_tokens;
    t.piece_sum = static_cast<uint64_t *>(workspace);
    t.nacc = nullptr;
    Recorder rec(opts);
    hipError_t e = rec.run(KID_BLOCK_WEIGHTS, stream, [&] { return launch_block_weights(t, stream); });
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "block weights launch: %s", hipGetErrorString(e));
    e = rec.run(KID_BLOCK_SELECT, stream, [&] { return launch_block_select(t, stream); });
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "block select launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

// ---- KV cache updates ----------------------------------------------------------

static spire_status check_new(const void *k_new, const void *v_new, int32_t new_dtype, int32_t D) {
    if (k_new == nullptr || v_new == nullptr) return fail(SPIRE_ERR_INVALID_ARG, "k_new or v_new is NULL");
    if (new_dtype != SPIRE_F32 && new_dtype != SPIRE_BF16)
        return fail(SPIRE_ERR_UNSUPPORTED, "new K/V must be F32 or BF16");
    const uintptr_t al = new_dtype == SPIRE_F32 ? 3u : 1u;
    if (((uintptr_t)k_new & al) != 0 || ((uintptr_t)v_new & al) != 0)
        return fail(SPIRE_ERR_INVALID_ARG, "new K/V must be aligned to their element size");
    if (D < 1 || D > 1024) return fail(SPIRE_ERR_UNSUPPORTED, "D must be in [1, 1024] (got %d)", D);
    return SPIRE_OK;
}

static bool elems_aligned(const spire_kv *kv) {
    const uintptr_t es = (uintptr_t)elem_size(kv->dtype);
    return es > 0 && ((uintptr_t)kv->k % es) == 0 && ((uintptr_t)kv->v % es) == 0;
}

spire_status spire_kv_append(const spire_kv *kv, const void *k_new, const void *v_new,
                             int32_t new_dtype, const int32_t *positions, int32_t B, int32_t Hkv,
                             int32_t D, int32_t T, hipStream_t stream) {
    g_err[0] = '\0';
    if (B < 0 || T < 0 || Hkv < 1) return fail(SPIRE_ERR_INVALID_ARG, "need B >= 0, T >= 0, Hkv >= 1");
    spire_status s = check_kv(kv, "kv", D, Hkv, true);
    if (s != SPIRE_OK) return s;
    if (B == 0 || T == 0) return SPIRE_OK;
    s = check_new(k_new, v_new, new_dtype, D);
    if (s != SPIRE_OK) return s;
    if (positions == nullptr) return fail(SPIRE_ERR_INVALID_ARG, "positions is NULL");
    if (!elems_aligned(kv)) return fail(SPIRE_ERR_INVALID_ARG, "kv storage not aligned to its element size");
    if ((int64_t)B * T * Hkv > ((int64_t)1 << 33)) return fail(SPIRE_ERR_UNSUPPORTED, "too many rows");
    const KvDev d = to_dev(kv);
    hipError_t e = launch_kv_append(d, k_new, v_new, new_dtype, positions, B, T, Hkv, D, stream);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "kv append launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

static spire_status check_draft_views(const spire_kv *sink, const spire_kv *ring, int32_t S, int32_t W,
                                      int32_t D, int32_t Hkv) {
    if (S < 0 || W < 0 || (int64_t)S + W < 1)
        return fail(SPIRE_ERR_INVALID_ARG, "need S >= 0, W >= 0, S + W >= 1 (S=%d, W=%d)", S, W);
    spire_status s = check_kv(sink, "sink", D, Hkv, false, S > 0);
    if (s != SPIRE_OK) return s;
    s = check_kv(ring, "ring", D, Hkv, false, W > 0);
    if (s != SPIRE_OK) return s;
    if (sink->dtype != ring->dtype) return fail(SPIRE_ERR_INVALID_ARG, "sink and ring dtypes differ");
    if (sink->capacity < S) return fail(SPIRE_ERR_INVALID_ARG, "sink capacity %d < S = %d", sink->capacity, S);
    if (ring->capacity < W) return fail(SPIRE_ERR_INVALID_ARG, "ring capacity %d < W = %d", ring->capacity, W);
    if ((S > 0 && !elems_aligned(sink)) || (W > 0 && !elems_aligned(ring)))
        return fail(SPIRE_ERR_INVALID_ARG, "sink/ring storage not aligned to its element size");
    return SPIRE_OK;
}

spire_status spire_draft_append(const spire_kv *sink, const spire_kv *ring, const void *k_new,
                                const void *v_new, int32_t new_dtype, const int32_t *seq_lens,
                                const int32_t *ring_offset, int32_t B, int32_t Hkv, int32_t D,
                                int32_t S, int32_t W, void *spill_k, void *spill_v,
                                hipStream_t stream) {
    g_err[0] = '\0';
    if (B < 0 || Hkv < 1) return fail(SPIRE_ERR_INVALID_ARG, "need B >= 0, Hkv >= 1");
    spire_status s = check_draft_views(sink, ring, S, W, D, Hkv);
    if (s != SPIRE_OK) return s;
    if (B == 0) return SPIRE_OK;
    s = check_new(k_new, v_new, new_dtype, D);
    if (s != SPIRE_OK) return s;
    if (seq_lens == nullptr || ring_offset == nullptr)
        return fail(SPIRE_ERR_INVALID_ARG, "seq_lens or ring_offset is NULL");
    if ((spill_k == nullptr) != (spill_v == nullptr))
        return fail(SPIRE_ERR_INVALID_ARG, "give both spill_k and spill_v, or neither");
    const KvDev ds = to_dev(sink), dr = to_dev(ring);
    hipError_t e = launch_draft_append(ds, dr, k_new, v_new, new_dtype, seq_lens, ring_offset, B, Hkv, D, S, W,
                                       spill_k, spill_v, stream);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "draft append launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

spire_status spire_draft_rollback(const spire_kv *sink, const spire_kv *ring, const void *spill_k,
                                  const void *spill_v, const int32_t *base_lens,
                                  const int32_t *n_accepted, int32_t steps,
                                  const int32_t *ring_offset, int32_t B, int32_t Hkv, int32_t D,
                                  int32_t S, int32_t W, hipStream_t stream) {
    g_err[0] = '\0';
    if (B < 0 || Hkv < 1 || steps < 0) return fail(SPIRE_ERR_INVALID_ARG, "need B >= 0, Hkv >= 1, steps >= 0");
    if (D < 1 || D > 1024) return fail(SPIRE_ERR_UNSUPPORTED, "D must be in [1, 1024] (got %d)", D);
    spire_status s = check_draft_views(sink, ring, S, W, D, Hkv);
    if (s != SPIRE_OK) return s;
    if (B == 0 || steps == 0) return SPIRE_OK;
    if (spill_k == nullptr || spill_v == nullptr || base_lens == nullptr || n_accepted == nullptr ||
        ring_offset == nullptr)
        return fail(SPIRE_ERR_INVALID_ARG, "spill_k, spill_v, base_lens, n_accepted or ring_offset is NULL");
    const KvDev ds = to_dev(sink), dr = to_dev(ring);
    hipError_t e = launch_draft_rollback(ds, dr, spill_k, spill_v, base_lens, n_accepted, steps, ring_offset, B,
                                         Hkv, D, S, W, stream);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "draft rollback launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

// ---- feedback memory -----------------------------------------------------------

spire_status spire_feedback_memory(const void *x, int32_t x_dtype, const float *w, int32_t n_out,
                                   int32_t layers, int32_t B, int32_t d, void *m, int32_t m_dtype,
                                   hipStream_t stream) {
    g_err[0] = '\0';
    if (n_out < 1 || n_out > kFmMaxOut)
        return fail(SPIRE_ERR_UNSUPPORTED, "n_out must be in [1, %d] (got %d)", kFmMaxOut, n_out);
    if (layers < 1 || layers > kFmMaxLayers)
        return fail(SPIRE_ERR_UNSUPPORTED, "layers must be in [1, %d] (got %d)", kFmMaxLayers, layers);
    if (B < 0 || d < 0) return fail(SPIRE_ERR_INVALID_ARG, "need B >= 0 and d >= 0");
    if ((x_dtype != SPIRE_F32 && x_dtype != SPIRE_BF16) || (m_dtype != SPIRE_F32 && m_dtype != SPIRE_BF16))
        return fail(SPIRE_ERR_UNSUPPORTED, "x and m must be F32 or BF16");
    if ((int64_t)B * d == 0) return SPIRE_OK;
    if (x == nullptr || w == nullptr || m == nullptr) return fail(SPIRE_ERR_INVALID_ARG, "x, w or m is NULL");
    const uintptr_t xa = x_dtype == SPIRE_F32 ? 3u : 1u, ma = m_dtype == SPIRE_F32 ? 3u : 1u;
    if (((uintptr_t)x & xa) != 0 || ((uintptr_t)m & ma) != 0 || ((uintptr_t)w & 3u) != 0)
        return fail(SPIRE_ERR_INVALID_ARG, "arrays must be aligned to their element size");
    FeedbackArgs a;
    a.x = x;
    a.w = w;
    a.m = m;
    a.x_dtype = x_dtype;
    a.m_dtype = m_dtype;
    a.n_out = n_out;
    a.Lp1 = layers;
    a.Bd = (int64_t)B * d;
    hipError_t e = launch_feedback_memory(a, stream);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "feedback memory launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

spire_status spire_hbm_read_probe(const void *buf, size_t bytes, uint32_t *sink, size_t sink_words,
                                  hipStream_t stream) {
    g_err[0] = '\0';
    if (sink == nullptr || (bytes > 0 && buf == nullptr)) return fail(SPIRE_ERR_INVALID_ARG, "buf or sink is NULL");
    if (sink_words < SPIRE_HBM_PROBE_SINK_WORDS)
        return fail(SPIRE_ERR_INVALID_ARG, "sink holds %zu words, needs %d", sink_words, SPIRE_HBM_PROBE_SINK_WORDS);
    if (((uintptr_t)buf & 15u) != 0 || bytes % 16 != 0)
        return fail(SPIRE_ERR_INVALID_ARG, "buf must be 16-byte aligned and bytes a multiple of 16");
    if (((uintptr_t)sink & 3u) != 0) return fail(SPIRE_ERR_INVALID_ARG, "sink must be 4-byte aligned");
    if (bytes > (size_t)INT64_MAX) return fail(SPIRE_ERR_INVALID_ARG, "bytes too large");
    hipError_t e = launch_hbm_read(buf, (int64_t)bytes, sink, stream);
    if (e != hipSuccess) return fail(SPIRE_ERR_HIP, "read probe launch: %s", hipGetErrorString(e));
    return SPIRE_OK;
}

}  // extern "C"
