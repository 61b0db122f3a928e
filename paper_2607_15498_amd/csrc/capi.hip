// C ABI of libvarrate: validation, sizing, workspace carving and kernel dispatch.
// Every check runs on the host before anything is enqueued; no entry point synchronises or
// allocates device memory.  The one piece of state kept across calls is the per (kernel,
// device) record of raised dynamic-LDS limits (ensure_lds_limit, under a lock).
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>

#include <map>
#include <mutex>
#include <string>
#include <utility>

#include "vr_internal.h"

using namespace vr;

namespace vr {

hipError_t ensure_lds_limit(const void* fn, size_t bytes) {
    static std::mutex mu;
    static std::map<std::pair<const void*, int>, size_t> raised;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    size_t& have = raised[{fn, dev}];
    if (bytes <= have) return hipSuccess;
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) have = bytes;
    return e;
}

}  // namespace vr

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return VARRATE_OK;
    return fail(VARRATE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }


int check_shape_only(const varrate_shape* sh) {
    if (!sh) return fail(VARRATE_EINVAL, "shape is NULL");
    if (sh->d != VARRATE_HEAD_DIM) return fail(VARRATE_EUNSUPPORTED, "head dim %d != 128", sh->d);
    if (sh->G < 1 || sh->H < 1) return fail(VARRATE_EINVAL, "G=%d H=%d must be >= 1", sh->G, sh->H);
    if (sh->H % sh->G != 0) return fail(VARRATE_EUNSUPPORTED, "H=%d is not a multiple of G=%d", sh->H, sh->G);
    if (sh->w < 1) return fail(VARRATE_EINVAL, "window w=%d must be >= 1", sh->w);
    if (sh->n <= sh->w) return fail(VARRATE_EBUDGET, "n=%lld leaves no coded tokens (w=%d)", (long long)sh->n, sh->w);
    if (sh->r_min < 0 || sh->r_min > VARRATE_HEAD_DIM)
        return fail(VARRATE_EINVAL, "r_min=%d outside [0, 128]", sh->r_min);
    if (sh->kappa_pct < 1 || sh->kappa_pct > 100) return fail(VARRATE_EINVAL, "kappa_pct=%d outside [1, 100]", sh->kappa_pct);
    if (sh->dtype != VARRATE_BF16 && sh->dtype != VARRATE_F32) return fail(VARRATE_EINVAL, "unknown dtype %d", sh->dtype);
    if ((int64_t)(sh->H / sh->G) * sh->w > 256)
        return fail(VARRATE_EUNSUPPORTED, "(H/G) * w = %lld window rows per KV head exceeds 256",
                    (long long)(sh->H / sh->G) * sh->w);
    if (sh->n - sh->w > MAX_CODED)
        return fail(VARRATE_EUNSUPPORTED, "N=%lld coded tokens exceeds %lld", (long long)(sh->n - sh->w), (long long)MAX_CODED);
    if (sh->anchor_stride != 0) {
        if (sh->anchor_stride < 2 || sh->anchor_stride > 4096)
            return fail(VARRATE_EINVAL, "anchor_stride=%d outside {0} or [2, 4096]", sh->anchor_stride);
        if (sh->dtype != VARRATE_BF16) return fail(VARRATE_EUNSUPPORTED, "the residual codec needs a bf16 layer");
        if (anchor_count(*sh) > 65535) return fail(VARRATE_EUNSUPPORTED, "more than 65535 anchors");
        if (anchor_count(*sh) < 4) return fail(VARRATE_EBUDGET, "fewer than 4 anchors");
        if (coded_count(*sh) < 1) return fail(VARRATE_EBUDGET, "no coded tokens between the anchors");
    }
    if (sh->rope != 0) {
        if (sh->rope != 1) return fail(VARRATE_EINVAL, "rope=%d outside {0, 1}", sh->rope);
        if (sh->anchor_stride != 0) return fail(VARRATE_EUNSUPPORTED, "rotary keys with anchors");
        for (int i = 0; i < VARRATE_HEAD_DIM / 2; ++i)
            if (!(sh->rope_theta[i] >= 0.f) || !std::isfinite(sh->rope_theta[i]))
                return fail(VARRATE_EINVAL, "rope_theta[%d] is negative or not finite", i);
    }
    return VARRATE_OK;
}

int check_shape(const varrate_shape* sh) {
    int rc = check_shape_only(sh);
    if (rc) return rc;
    const int64_t B = coded_budget(*sh);
    const int64_t N = coded_count(*sh);
    if (N * sh->r_min > B || B > N * VARRATE_HEAD_DIM)
        return fail(VARRATE_EBUDGET, "budget B=%lld infeasible for N=%lld, r_min=%d, R=128", (long long)B,
                    (long long)N, sh->r_min);
    return VARRATE_OK;
}

// shared cross-head basis: R rows, joint budget
int64_t joint_budget(const varrate_shape& sh) {
    return varrate_coded_budget(sh.n, 2 * sh.G * VARRATE_HEAD_DIM, sh.w, sh.kappa_pct);
}

int check_joint(const varrate_shape* sh, int R) {
    int rc = check_shape_only(sh);
    if (rc) return rc;
    if (sh->rope || sh->anchor_stride)
        return fail(VARRATE_EUNSUPPORTED, "the shared basis takes position-free keys and no anchors");
    const int Dz = 2 * sh->G * VARRATE_HEAD_DIM;
    if (R < 256 || R > 1024 || R % 256 != 0 || R > Dz)
        return fail(VARRATE_EUNSUPPORTED, "R=%d: need a multiple of 256 in [256, min(1024, 2 G d = %d)]", R, Dz);
    if (sh->r_min > R) return fail(VARRATE_EINVAL, "r_min=%d exceeds R=%d", sh->r_min, R);
    const int64_t B = joint_budget(*sh);
    const int64_t N = sh->n - sh->w;
    if (N * sh->r_min > B || B > N * R)
        return fail(VARRATE_EBUDGET, "joint budget B=%lld infeasible for N=%lld, r_min=%d, R=%d", (long long)B,
                    (long long)N, sh->r_min, R);
    if (B + VARRATE_JOINT_PAD > (int64_t)UINT32_MAX)
        return fail(VARRATE_EUNSUPPORTED, "joint budget B=%lld exceeds 32-bit offsets", (long long)B);
    return VARRATE_OK;
}

int check_jcache(const varrate_shape* sh, const varrate_jcache* c) {
    if (!c) return fail(VARRATE_EINVAL, "jcache is NULL");
    int rc = check_joint(sh, c->R);
    if (rc) return rc;
    if (!c->coef || !c->rank || !c->offset || !c->chunk_off || !c->k_exact || !c->v_exact)
        return fail(VARRATE_EINVAL, "jcache has a NULL buffer");
    if (!aligned16(c->coef) || !aligned16(c->k_exact) || !aligned16(c->v_exact))
        return fail(VARRATE_EINVAL, "jcache buffers must be 16-byte aligned");
    if (c->coef_stride < joint_budget(*sh) + VARRATE_JOINT_PAD)
        return fail(VARRATE_EINVAL, "coef_stride %lld < B + %d", (long long)c->coef_stride, VARRATE_JOINT_PAD);
    if (c->cap < sh->w || c->cap > 8192) return fail(VARRATE_EINVAL, "exact capacity %lld outside [w, 8192]",
                                                     (long long)c->cap);
    return VARRATE_OK;
}

int check_cache(const varrate_shape* sh, const varrate_cache* c, bool need_layout) {
    if (!c) return fail(VARRATE_EINVAL, "cache is NULL");
    const int64_t B = coded_budget(*sh);
    if (sh->anchor_stride != 0 && (!c->k_anchor || !c->v_anchor || !c->snn || !c->inv_off || !c->inv_pos ||
                                   !c->piece_off || !c->piece_anchor))
        return fail(VARRATE_EINVAL, "cache has a NULL anchor buffer");
    if (sh->anchor_stride != 0 && (!aligned16(c->k_anchor) || !aligned16(c->v_anchor)))
        return fail(VARRATE_EINVAL, "anchor buffers must be 16-byte aligned");
    if (!c->coef_k || !c->coef_v || !c->rank || !c->chunk_off || !c->k_exact || !c->v_exact ||
        (need_layout && (!c->srank || !c->sidx)))
        return fail(VARRATE_EINVAL, "cache has a NULL buffer");
    if (!aligned16(c->coef_k) || !aligned16(c->coef_v) || !aligned16(c->k_exact) || !aligned16(c->v_exact))
        return fail(VARRATE_EINVAL, "cache buffers must be 16-byte aligned");
    const int64_t N = coded_count(*sh);
    const int64_t need = B + (int64_t)8 * VARRATE_CHUNK * ((N + VARRATE_CHUNK - 1) / VARRATE_CHUNK) + VARRATE_COEF_PAD;
    if (c->coef_stride < need || (c->coef_stride % 8) != 0)
        return fail(VARRATE_EINVAL, "coef_stride=%lld must be a multiple of 8 and >= %lld (B + 2048 per chunk + %d)",
                    (long long)c->coef_stride, (long long)need, VARRATE_COEF_PAD);
    if (c->cap < sh->w) return fail(VARRATE_EINVAL, "exact capacity %lld < w=%d", (long long)c->cap, sh->w);
    return VARRATE_OK;
}

size_t compress_ws_base(const varrate_shape& sh) {
    const int64_t N = sh.n - sh.w;
    return align256(salience_ws_bytes(sh)) + align256(allocate_ws_bytes(sh)) + align256((size_t)N * 4);
}

// rotary keys: the un-rotated copy of K [n][G][d] follows the other buffers
size_t compress_ws(const varrate_shape& sh) {
    if (sh.anchor_stride != 0) return anchor_ws_bytes(sh);
    const size_t es = sh.dtype == VARRATE_BF16 ? 2 : 4;
    return compress_ws_base(sh) + (sh.rope ? align256((size_t)sh.n * sh.G * VARRATE_HEAD_DIM * es) : 0);
}

// Eq. (6) projection; with rotary keys, of the keys turned back to pre-RoPE (Algorithm 1,
// first step) in the workspace
// chunk_sizes: as launch_project's (NULL: the cache's chunk table is already scanned)
hipError_t project_keys(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                        const float* PV, varrate_cache& c, uint8_t* ws, hipStream_t st,
                        const uint32_t* chunk_sizes = nullptr) {
    if (!sh.rope) return launch_project(sh, K, V, PK, PV, c, st, chunk_sizes);
    void* Kr = ws + compress_ws_base(sh);
    hipError_t e = launch_rope_unrotate(sh, K, Kr, st);
    if (e != hipSuccess) return e;
    return launch_project(sh, Kr, V, PK, PV, c, st, chunk_sizes);
}

}  // namespace

extern "C" {

const char* varrate_status_string(int s) {
    switch (s) {
        case VARRATE_OK: return "ok";
        case VARRATE_EINVAL: return "invalid argument";
        case VARRATE_EBUDGET: return "infeasible budget";
        case VARRATE_EUNSUPPORTED: return "unsupported shape";
        case VARRATE_EHIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char* varrate_last_error(void) { return g_err.c_str(); }

int varrate_version(void) { return 1; }

int varrate_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream) {
    if (!src || !sink || !aligned16(src) || bytes == 0 || bytes % 16 != 0)
        return fail(VARRATE_EINVAL, "read probe: src and sink non-NULL, src 16-byte aligned, bytes a positive "
                                    "multiple of 16");
    return hip_status(launch_read_probe(src, bytes, sink, (hipStream_t)stream), "read probe launch");
}

int64_t varrate_coded_budget(int64_t n, int32_t d, int32_t w, int32_t kappa_pct) {
    return ((int64_t)kappa_pct * n * d) / 100 - (int64_t)w * d;
}

int varrate_cache_bytes(const varrate_shape* sh, int64_t cap, varrate_cache_bytes_t* out) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (!out) return fail(VARRATE_EINVAL, "out is NULL");
    if (cap < sh->w) return fail(VARRATE_EINVAL, "exact capacity %lld < w=%d", (long long)cap, sh->w);
    const size_t es = sh->dtype == VARRATE_BF16 ? 2 : 4;
    out->N = coded_count(*sh);
    out->B = coded_budget(*sh);
    out->na = anchor_count(*sh);
    out->k_anchor = out->v_anchor = (size_t)out->na * sh->G * VARRATE_HEAD_DIM * es;
    out->snn = out->na ? (size_t)out->N * 4 * 2 : 0;
    out->inv_off = out->na ? (size_t)(out->na + 1) * 4 : 0;
    out->inv_pos = out->na ? (size_t)out->N * 4 * 4 : 0;
    out->piece_off = out->inv_off;
    out->piece_anchor = out->na ? (size_t)(out->N * 4 / 64 + out->na) * 2 : 0;
    out->n_chunks = (out->N + VARRATE_CHUNK - 1) / VARRATE_CHUNK;
    // tile rectangles: a chunk's 16 tiles take at most its ranks + 16 x 128 elements
    const int64_t bound = out->B + (int64_t)8 * VARRATE_CHUNK * out->n_chunks;
    out->coef_stride = ((bound + VARRATE_COEF_PAD + 63) / 64) * 64;
    out->coef_k = out->coef_v = (size_t)sh->G * out->coef_stride * es;
    out->rank = out->srank = (size_t)((out->N + 63) / 64) * 64;   // padded for 16-byte loads
    out->sidx = (size_t)out->N * 4;
    out->chunk_off = (size_t)(out->n_chunks + 1) * 4;
    out->k_exact = out->v_exact = (size_t)sh->G * cap * VARRATE_HEAD_DIM * es;
    return VARRATE_OK;
}

size_t varrate_compress_workspace_bytes(const varrate_shape* sh) {
    if (check_shape(sh)) return 0;
    return compress_ws(*sh);
}

size_t varrate_decode_workspace_bytes(const varrate_shape* sh, int32_t S, int32_t Q) {
    if (check_shape(sh) || S < 1 || Q < 1) return 0;
    return decode_ws_bytes(*sh, S, Q);
}

static int ws_check(void* ws, size_t have, size_t need) {
    if (!ws) return fail(VARRATE_EINVAL, "workspace is NULL");
    if (!aligned16(ws)) return fail(VARRATE_EINVAL, "workspace must be 16-byte aligned");
    if (have < need) return fail(VARRATE_EINVAL, "workspace %zu bytes < required %zu", have, need);
    return VARRATE_OK;
}

int varrate_salience(const varrate_shape* sh, const void* K, const void* Qw, float* sbar, void* ws,
                     size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (!K || !Qw || !sbar) return fail(VARRATE_EINVAL, "K, Qw and sbar must be non-NULL");
    if (!aligned16(K) || !aligned16(Qw)) return fail(VARRATE_EINVAL, "K and Qw must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    return hip_status(launch_salience(*sh, K, Qw, sbar, (uint8_t*)ws, (hipStream_t)stream), "salience launch");
}

int varrate_allocate(const varrate_shape* sh, const float* sbar, varrate_cache* c, void* ws,
                     size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (sh->anchor_stride) return fail(VARRATE_EUNSUPPORTED, "residual codec: use varrate_anchor_encode");
    if ((rc = check_cache(sh, c, false))) return rc;
    if (!sbar) return fail(VARRATE_EINVAL, "sbar is NULL");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    c->N = sh->n - sh->w;
    c->B = varrate_coded_budget(sh->n, sh->d, sh->w, sh->kappa_pct);
    uint8_t* w8 = (uint8_t*)ws + align256(salience_ws_bytes(*sh));
    return hip_status(launch_allocate(*sh, sbar, *c, w8, (hipStream_t)stream), "allocate launch");
}

int varrate_project(const varrate_shape* sh, const void* K, const void* V, const float* PK,
                    const float* PV, varrate_cache* c, void* ws, size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (sh->anchor_stride) return fail(VARRATE_EUNSUPPORTED, "residual codec: use varrate_anchor_encode");
    if ((rc = check_cache(sh, c, true))) return rc;
    if (!K || !V || !PK || !PV) return fail(VARRATE_EINVAL, "K, V, P_K and P_V must be non-NULL");
    if (!aligned16(K) || !aligned16(V) || !aligned16(PK) || !aligned16(PV))
        return fail(VARRATE_EINVAL, "K, V, P_K, P_V must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    c->N = sh->n - sh->w;
    c->B = varrate_coded_budget(sh->n, sh->d, sh->w, sh->kappa_pct);
    hipStream_t st = (hipStream_t)stream;
    rc = hip_status(project_keys(*sh, K, V, PK, PV, *c, (uint8_t*)ws, st), "project launch");
    if (rc) return rc;
    c->n_exact = sh->w;
    return VARRATE_OK;
}

int varrate_compress(const varrate_shape* sh, const void* K, const void* V, const void* Qw,
                     const float* PK, const float* PV, varrate_cache* c, float* sbar_out, void* ws,
                     size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if ((rc = check_cache(sh, c, true))) return rc;
    if (!K || !V || !Qw || !PK || !PV) return fail(VARRATE_EINVAL, "inputs must be non-NULL");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    if (!aligned16(K) || !aligned16(V) || !aligned16(Qw) || !aligned16(PK) || !aligned16(PV))
        return fail(VARRATE_EINVAL, "K, V, Qw, P_K, P_V must be 16-byte aligned");
    if (sh->anchor_stride) {
        // residual codec: salience over the whole prefix (pooled), anchor search, encode
        hipStream_t st = (hipStream_t)stream;
        const AnchorWs w = anchor_ws(*sh, (uint8_t*)ws);
        float* sb = sbar_out ? sbar_out : w.sbar;
        if ((rc = hip_status(launch_salience(*sh, K, Qw, sb, w.sal, st, true), "salience launch"))) return rc;
        if ((rc = hip_status(launch_anchor_search(*sh, K, V, w.nn, w, st), "anchor search launch"))) return rc;
        c->N = coded_count(*sh);
        c->B = coded_budget(*sh);
        c->na = anchor_count(*sh);
        if ((rc = hip_status(launch_anchor_encode(*sh, K, V, sb, w.nn, PK, PV, *c, w, st), "anchor encode launch")))
            return rc;
        c->n_exact = sh->w;
        return VARRATE_OK;
    }
    float* sbar = sbar_out;
    if (!sbar) {
        sbar = (float*)((uint8_t*)ws + align256(salience_ws_bytes(*sh)) + align256(allocate_ws_bytes(*sh)));
    }
    // salience passes, then the allocation's first pass pools sbar from the column sums
    // itself (the separate pooling launch is skipped), then the rest of the allocation and
    // the projection, which scans the chunk sizes into the chunk table itself (the
    // allocation's scan launch is skipped): the same results as the three entry points in turn
    hipStream_t st = (hipStream_t)stream;
    uint8_t* w0 = (uint8_t*)ws;
    if ((rc = hip_status(launch_salience(*sh, K, Qw, sbar, w0, st, false), "salience launch"))) return rc;
    c->N = sh->n - sh->w;
    c->B = varrate_coded_budget(sh->n, sh->d, sh->w, sh->kappa_pct);
    uint8_t* w8 = w0 + align256(salience_ws_bytes(*sh));
    const uint32_t* csz = nullptr;
    if ((rc = hip_status(launch_allocate(*sh, sbar, *c, w8, st, salience_part(*sh, w0), &csz), "allocate launch")))
        return rc;
    if ((rc = hip_status(project_keys(*sh, K, V, PK, PV, *c, w0, st, csz), "project launch"))) return rc;
    c->n_exact = sh->w;
    return VARRATE_OK;
}

int varrate_anchor_search(const varrate_shape* sh, const void* K, const void* V, uint16_t* nn, void* ws,
                          size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (!sh->anchor_stride) return fail(VARRATE_EINVAL, "anchor_stride is 0");
    if (!K || !V || !nn) return fail(VARRATE_EINVAL, "K, V and nn must be non-NULL");
    if (!aligned16(K) || !aligned16(V)) return fail(VARRATE_EINVAL, "K and V must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    const AnchorWs w = anchor_ws(*sh, (uint8_t*)ws);
    return hip_status(launch_anchor_search(*sh, K, V, nn, w, (hipStream_t)stream), "anchor search launch");
}

int varrate_anchor_encode(const varrate_shape* sh, const void* K, const void* V, const float* sbar, const uint16_t* nn,
                          const float* PK, const float* PV, varrate_cache* c, void* ws, size_t ws_bytes, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (!sh->anchor_stride) return fail(VARRATE_EINVAL, "anchor_stride is 0");
    if ((rc = check_cache(sh, c, true))) return rc;
    if (!K || !V || !sbar || !nn || !PK || !PV) return fail(VARRATE_EINVAL, "inputs must be non-NULL");
    if (!aligned16(K) || !aligned16(V) || !aligned16(PK) || !aligned16(PV))
        return fail(VARRATE_EINVAL, "K, V, P_K, P_V must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, compress_ws(*sh)))) return rc;
    const AnchorWs w = anchor_ws(*sh, (uint8_t*)ws);
    c->N = coded_count(*sh);
    c->B = coded_budget(*sh);
    c->na = anchor_count(*sh);
    if ((rc = hip_status(launch_anchor_encode(*sh, K, V, sbar, nn, PK, PV, *c, w, (hipStream_t)stream),
                         "anchor encode launch")))
        return rc;
    c->n_exact = sh->w;
    return VARRATE_OK;
}

int varrate_append_exact(const varrate_shape* sh, varrate_cache* c, const void* k_new, const void* v_new,
                         void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if ((rc = check_cache(sh, c, false))) return rc;
    if (!k_new || !v_new) return fail(VARRATE_EINVAL, "k_new and v_new must be non-NULL");
    if (c->n_exact >= c->cap) return fail(VARRATE_EINVAL, "exact capacity %lld is full", (long long)c->cap);
    const size_t es = sh->dtype == VARRATE_BF16 ? 2 : 4;
    const size_t row = VARRATE_HEAD_DIM * es;
    hipStream_t st = (hipStream_t)stream;
    for (int kv = 0; kv < 2; ++kv) {
        uint8_t* dst = (uint8_t*)(kv ? c->v_exact : c->k_exact) + (size_t)c->n_exact * row;
        const void* src = kv ? v_new : k_new;
        hipError_t e = hipMemcpy2DAsync(dst, (size_t)c->cap * row, src, row, row, sh->G,
                                        hipMemcpyDeviceToDevice, st);
        if ((rc = hip_status(e, "append copy"))) return rc;
    }
    c->n_exact += 1;
    return VARRATE_OK;
}

static int check_decode(const varrate_shape* sh, const varrate_cache* caches, int32_t S, const void* q,
                        int32_t Q, const float* PK, const float* PV, void* out) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (!caches || S < 1 || S > VARRATE_MAX_SEQS) return fail(VARRATE_EINVAL, "S=%d outside [1, %d]", S, VARRATE_MAX_SEQS);
    if (Q < 1 || (int64_t)Q * (sh->H / sh->G) > VARRATE_MAX_QROWS)
        return fail(VARRATE_EUNSUPPORTED, "Q=%d query rows per KV head exceed %d", Q, VARRATE_MAX_QROWS);
    if (!q || !out || !PK || !PV) return fail(VARRATE_EINVAL, "q, out, P_K, P_V must be non-NULL");
    if (!aligned16(q) || !aligned16(PK) || !aligned16(PV))
        return fail(VARRATE_EINVAL, "q, P_K, P_V must be 16-byte aligned");
    for (int s = 0; s < S; ++s) {
        if ((rc = check_cache(sh, &caches[s], true))) return rc;
        if (caches[s].N != coded_count(*sh)) return fail(VARRATE_EINVAL, "cache %d was not compressed with this shape", s);
        if (caches[s].n_exact < 0 || caches[s].n_exact > caches[s].cap)
            return fail(VARRATE_EINVAL, "cache %d has n_exact outside [0, cap]", s);
        if (caches[s].coef_stride != caches[0].coef_stride || caches[s].cap != caches[0].cap)
            return fail(VARRATE_EINVAL, "caches must share coef_stride and cap");
    }
    if (!decode_supported(*sh, S, Q))
        return fail(VARRATE_EUNSUPPORTED, "S * G * ceil(Q H/G / 16) exceeds 16384 merge slots");
    return VARRATE_OK;
}

int varrate_decode_attn(const varrate_shape* sh, const varrate_cache* caches, int32_t S, const void* q,
                        int32_t Q, const float* PK, const float* PV, void* out, void* ws, size_t ws_bytes,
                        void* stream) {
    int rc = check_decode(sh, caches, S, q, Q, PK, PV, out);
    if (rc) return rc;
    if ((rc = ws_check(ws, ws_bytes, decode_ws_bytes(*sh, S, Q)))) return rc;
    return hip_status(launch_decode(*sh, caches, S, q, Q, PK, PV, out, (uint8_t*)ws, (hipStream_t)stream),
                      "decode launch");
}

int varrate_qcache_bytes(const varrate_shape* sh, int32_t bits, int64_t* q_stride, size_t* qchunk_off_bytes) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (bits != 3 && bits != 4 && bits != 8) return fail(VARRATE_EUNSUPPORTED, "bits=%d not in {3, 4, 8}", bits);
    if (!q_stride || !qchunk_off_bytes) return fail(VARRATE_EINVAL, "outputs must be non-NULL");
    const int64_t N = coded_count(*sh);
    *q_stride = (int64_t)qcache_stride(*sh, bits);
    *qchunk_off_bytes = (size_t)((N + VARRATE_CHUNK - 1) / VARRATE_CHUNK + 1) * 4;
    return VARRATE_OK;
}

static int check_qcache(const varrate_shape* sh, const varrate_qcache* q) {
    if (!q) return fail(VARRATE_EINVAL, "qcache is NULL");
    if (sh->dtype != VARRATE_BF16) return fail(VARRATE_EUNSUPPORTED, "quantised coefficients need a bf16 layer");
    if (q->bits != 3 && q->bits != 4 && q->bits != 8)
        return fail(VARRATE_EUNSUPPORTED, "bits=%d not in {3, 4, 8}", q->bits);
    if (!q->code_k || !q->code_v || !q->qchunk_off) return fail(VARRATE_EINVAL, "qcache has a NULL buffer");
    if (!aligned16(q->code_k) || !aligned16(q->code_v)) return fail(VARRATE_EINVAL, "code buffers must be 16-byte aligned");
    const int64_t need = (int64_t)qcache_stride(*sh, q->bits);
    if (q->q_stride < need || (q->q_stride % 16) != 0)
        return fail(VARRATE_EINVAL, "q_stride=%lld must be a multiple of 16 and >= %lld", (long long)q->q_stride,
                    (long long)need);
    return VARRATE_OK;
}

int varrate_quantize(const varrate_shape* sh, const varrate_cache* c, varrate_qcache* q, void* stream) {
    int rc = check_shape(sh);
    if (rc) return rc;
    if (sh->rope) return fail(VARRATE_EUNSUPPORTED, "quantised coefficients of rotary keys");
    if ((rc = check_cache(sh, c, true))) return rc;
    if ((rc = check_qcache(sh, q))) return rc;
    return hip_status(launch_quantize(*sh, *c, *q, (hipStream_t)stream), "quantize launch");
}

int varrate_decode_attn_q(const varrate_shape* sh, const varrate_cache* caches, const varrate_qcache* qcaches,
                          int32_t S, const void* q, int32_t Q, const float* PK, const float* PV, void* out,
                          void* ws, size_t ws_bytes, void* stream) {
    int rc = check_decode(sh, caches, S, q, Q, PK, PV, out);
    if (rc) return rc;
    if (sh->rope) return fail(VARRATE_EUNSUPPORTED, "quantised coefficients of rotary keys");
    if (!qcaches) return fail(VARRATE_EINVAL, "qcaches is NULL");
    for (int s = 0; s < S; ++s) {
        if ((rc = check_qcache(sh, &qcaches[s]))) return rc;
        if (qcaches[s].bits != qcaches[0].bits || qcaches[s].q_stride != qcaches[0].q_stride)
            return fail(VARRATE_EINVAL, "qcaches must share bits and q_stride");
    }
    if ((rc = ws_check(ws, ws_bytes, decode_ws_bytes(*sh, S, Q)))) return rc;
    return hip_status(launch_decode(*sh, caches, S, q, Q, PK, PV, out, (uint8_t*)ws, (hipStream_t)stream, false,
                                    qcaches),
                      "decode launch");
}

int varrate_jcache_bytes(const varrate_shape* sh, int32_t R, int64_t cap, varrate_jcache_bytes_t* out) {
    int rc = check_joint(sh, R);
    if (rc) return rc;
    if (!out) return fail(VARRATE_EINVAL, "out is NULL");
    if (cap < sh->w || cap > 8192) return fail(VARRATE_EINVAL, "exact capacity %lld outside [w, 8192]", (long long)cap);
    const size_t es = sh->dtype == VARRATE_BF16 ? 2 : 4;
    out->N = sh->n - sh->w;
    out->B = joint_budget(*sh);
    out->n_chunks = (out->N + VARRATE_CHUNK - 1) / VARRATE_CHUNK;
    out->coef_stride = ((out->B + VARRATE_JOINT_PAD + 63) / 64) * 64;
    out->coef = (size_t)out->coef_stride * es;
    out->rank = (size_t)((out->N + 31) / 32) * 64;
    out->offset = (size_t)(out->N + 1) * 4;
    out->chunk_off = (size_t)(out->n_chunks + 1) * 4;
    out->k_exact = out->v_exact = (size_t)sh->G * cap * VARRATE_HEAD_DIM * es;
    return VARRATE_OK;
}

size_t varrate_joint_compress_workspace_bytes(const varrate_shape* sh, int32_t R) {
    if (check_joint(sh, R)) return 0;
    return compress_ws_base(*sh);
}

size_t varrate_joint_decode_workspace_bytes(const varrate_shape* sh, int32_t R, int32_t S, int32_t Q) {
    if (check_joint(sh, R) || S < 1 || Q < 1 || (int64_t)Q * sh->H > 32) return 0;
    return joint_decode_ws_bytes(*sh, R, S, Q);
}

int varrate_joint_compress(const varrate_shape* sh, const void* K, const void* V, const void* Qw, const float* W,
                           varrate_jcache* c, float* sbar_out, void* ws, size_t ws_bytes, void* stream) {
    int rc = check_jcache(sh, c);
    if (rc) return rc;
    if (!K || !V || !Qw || !W) return fail(VARRATE_EINVAL, "inputs must be non-NULL");
    if (!aligned16(K) || !aligned16(V) || !aligned16(Qw) || !aligned16(W))
        return fail(VARRATE_EINVAL, "K, V, Qw, W must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, compress_ws_base(*sh)))) return rc;
    hipStream_t st = (hipStream_t)stream;
    uint8_t* w0 = (uint8_t*)ws;
    float* sbar = sbar_out ? sbar_out
                           : (float*)(w0 + align256(salience_ws_bytes(*sh)) + align256(allocate_ws_bytes(*sh)));
    c->N = sh->n - sh->w;
    c->B = joint_budget(*sh);
    if ((rc = hip_status(launch_salience(*sh, K, Qw, sbar, w0, st, false), "salience launch"))) return rc;
    uint8_t* w8 = w0 + align256(salience_ws_bytes(*sh));
    if ((rc = hip_status(launch_allocate_joint(*sh, c->R, c->B, sbar, c->rank, c->offset, c->chunk_off, w8, st,
                                               salience_part(*sh, w0)),
                         "allocate launch")))
        return rc;
    if ((rc = hip_status(launch_joint_project(*sh, c->R, K, V, W, c->rank, c->offset, c->coef, st), "project launch")))
        return rc;
    if ((rc = hip_status(launch_joint_window(*sh, K, V, *c, st), "window copy"))) return rc;
    c->n_exact = sh->w;
    return VARRATE_OK;
}

int varrate_joint_decode_attn(const varrate_shape* sh, const varrate_jcache* caches, int32_t S, const void* q,
                              int32_t Q, const float* W, void* out, void* ws, size_t ws_bytes, void* stream) {
    if (!caches || S < 1 || S > VARRATE_MAX_SEQS) return fail(VARRATE_EINVAL, "S=%d outside [1, %d]", S, VARRATE_MAX_SEQS);
    int rc;
    for (int s = 0; s < S; ++s) {
        if ((rc = check_jcache(sh, &caches[s]))) return rc;
        if (caches[s].N != sh->n - sh->w || caches[s].R != caches[0].R || caches[s].cap != caches[0].cap)
            return fail(VARRATE_EINVAL, "jcache %d does not match the shape, R or cap of jcache 0", s);
        if (caches[s].n_exact < 1 || caches[s].n_exact > caches[s].cap)
            return fail(VARRATE_EINVAL, "jcache %d has n_exact outside [1, cap]", s);
    }
    if (Q < 1 || (int64_t)Q * sh->H > 32) return fail(VARRATE_EUNSUPPORTED, "Q H = %lld query rows exceed 32",
                                                      (long long)Q * sh->H);
    if (!q || !out || !W) return fail(VARRATE_EINVAL, "q, out and W must be non-NULL");
    if (!aligned16(q) || !aligned16(W)) return fail(VARRATE_EINVAL, "q and W must be 16-byte aligned");
    if ((rc = ws_check(ws, ws_bytes, joint_decode_ws_bytes(*sh, caches[0].R, S, Q)))) return rc;
    return hip_status(launch_joint_decode(*sh, caches[0].R, caches, S, q, Q, W, out, (uint8_t*)ws,
                                          (hipStream_t)stream),
                      "joint decode launch");
}

int varrate_joint_append_exact(const varrate_shape* sh, varrate_jcache* c, const void* k_new, const void* v_new,
                               void* stream) {
    int rc = check_jcache(sh, c);
    if (rc) return rc;
    if (!k_new || !v_new) return fail(VARRATE_EINVAL, "k_new and v_new must be non-NULL");
    if (c->n_exact >= c->cap) return fail(VARRATE_EINVAL, "exact capacity %lld is full", (long long)c->cap);
    const size_t es = sh->dtype == VARRATE_BF16 ? 2 : 4;
    const size_t row = VARRATE_HEAD_DIM * es;
    hipStream_t st = (hipStream_t)stream;
    for (int kv = 0; kv < 2; ++kv) {
        uint8_t* dst = (uint8_t*)(kv ? c->v_exact : c->k_exact) + (size_t)c->n_exact * row;
        const void* src = kv ? v_new : k_new;
        hipError_t e = hipMemcpy2DAsync(dst, (size_t)c->cap * row, src, row, row, sh->G, hipMemcpyDeviceToDevice, st);
        if ((rc = hip_status(e, "append copy"))) return rc;
    }
    c->n_exact += 1;
    return VARRATE_OK;
}

size_t varrate_decode_scratch_need(const varrate_shape* sh, int32_t S, int32_t Q) {
    if (check_shape(sh) || S < 1 || S > VARRATE_MAX_SEQS || Q < 1 ||
        (int64_t)Q * (sh->H / sh->G) > VARRATE_MAX_QROWS)
        return 0;
    return decode_group_bytes(*sh, S, Q);
}

int varrate_decode_attn_noalloc(const varrate_shape* sh, const varrate_cache* caches, int32_t S, const void* q,
                                int32_t Q, const float* PK, const float* PV, void* out, void* stream) {
    int rc = check_decode(sh, caches, S, q, Q, PK, PV, out);
    if (rc) return rc;
    if (sh->anchor_stride || sh->rope)
        return fail(VARRATE_EUNSUPPORTED, "the residual codec's and rotary keys' decode need a workspace "
                                          "(varrate_decode_attn)");
    const size_t need = decode_group_bytes(*sh, S, Q);
    if (need > (size_t)VARRATE_DECODE_SCRATCH_BYTES)
        return fail(VARRATE_EUNSUPPORTED,
                    "this decode needs %zu bytes of partial records, more than the fixed %zu-byte scratch; "
                    "call varrate_decode_attn with a workspace instead",
                    need, (size_t)VARRATE_DECODE_SCRATCH_BYTES);
    uint8_t* scratch = nullptr;
    if ((rc = hip_status(decode_scratch(&scratch), "decode scratch lookup"))) return rc;
    return hip_status(launch_decode(*sh, caches, S, q, Q, PK, PV, out, scratch, (hipStream_t)stream, true),
                      "decode launch");
}

}  // extern "C"
