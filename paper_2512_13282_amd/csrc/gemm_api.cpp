// gemm_api.cpp -- the C ABI entry points (host side).
//
// Validation happens here, on the host, before any HIP call; the plan comes
// from the selector (cached per shape/alignment class); the launch goes
// through launch_gemm (gemm_launch.hip).
#include <errno.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/gemm_mi355x.h"
#include "configs.h"
#include "launch.h"
#include "selector.h"

namespace {

using gemm::Plan;
using gemm::Problem;

struct Override {
    int32_t family = -1;   // -1 = automatic
    int32_t config = -1;
    int32_t split = 0;
    int32_t reduce = -1;   // -1 = automatic
};

std::mutex g_mu;
Override g_override[2];

struct Key {
    int32_t dtype;
    int64_t M, N, K;
    bool vec;
    int32_t trans_b;
    bool operator==(const Key &o) const {
        return dtype == o.dtype && M == o.M && N == o.N && K == o.K && vec == o.vec && trans_b == o.trans_b;
    }
};
// 64-bit FNV-1a over the key's fields (its published offset basis and prime).
struct KeyHash {
    size_t operator()(const Key &k) const {
        uint64_t h = 1469598103934665603ULL;
        auto mix = [&](uint64_t v) { h = (h ^ v) * 1099511628211ULL; };
        mix(uint64_t(k.dtype)); mix(uint64_t(k.M)); mix(uint64_t(k.N)); mix(uint64_t(k.K));
        mix(uint64_t(k.vec)); mix(uint64_t(k.trans_b));
        return size_t(h);
    }
};
struct CachedPlan {
    Plan plan;
    int32_t source;   // GEMM_PLAN_FROM_*
};
std::unordered_map<Key, CachedPlan, KeyHash> g_cache;

// Plans loaded at run time (gemm_load_plans, GEMM_MI355X_PLANS), per exact shape and
// B layout; they take precedence over the compiled table.  Guarded by g_mu.
struct Shape {
    int32_t dtype;
    int64_t M, N, K;
    int32_t trans_b;
    bool operator==(const Shape &o) const {
        return dtype == o.dtype && M == o.M && N == o.N && K == o.K && trans_b == o.trans_b;
    }
};
struct ShapeHash {
    size_t operator()(const Shape &s) const { return KeyHash()(Key{s.dtype, s.M, s.N, s.K, false, s.trans_b}); }
};
struct LoadedPlan {
    int32_t config, split, reduce;
};
std::unordered_map<Shape, LoadedPlan, ShapeHash> g_loaded;
std::once_flag g_env_once;

// One field of a plan line: a decimal integer in [lo, hi].  Advances *s past it.
bool parse_field(char **s, long long lo, long long hi, long long *v) {
    char *end = nullptr;
    errno = 0;
    const long long x = strtoll(*s, &end, 10);
    if (end == *s || errno != 0 || x < lo || x > hi) return false;
    *v = x;
    *s = end;
    return true;
}

// Reads a plan file: one plan per line, "dtype M N K config split reduce trans_b" (the
// fields of the compiled table), '#' to the end of a line is a comment, blank lines
// are skipped, lines are at most 510 characters.  An unreadable file or a malformed,
// out-of-range or overlong line returns GEMM_ERR_INVALID_VALUE, and the caller then
// loads none of the file.
int read_plan_file(const char *path, std::vector<std::pair<Shape, LoadedPlan>> *out) {
    if (path == nullptr) return GEMM_ERR_INVALID_VALUE;
    FILE *f = fopen(path, "r");
    if (f == nullptr) return GEMM_ERR_INVALID_VALUE;
    const long long kMaxDim = 1LL << 55;
    char line[512];
    int rc = GEMM_OK;
    while (rc == GEMM_OK && fgets(line, sizeof(line), f) != nullptr) {
        if (strchr(line, '\n') == nullptr && !feof(f)) { rc = GEMM_ERR_INVALID_VALUE; break; }   // too long
        if (char *hash = strchr(line, '#')) *hash = '\0';
        char *s = line;
        while (*s == ' ' || *s == '\t' || *s == '\r' || *s == '\n') ++s;
        if (*s == '\0') continue;
        long long v[8];
        const long long lo[8] = {0, 0, 0, 0, 0, 1, -1, 0};
        const long long hi[8] = {1, kMaxDim, kMaxDim, kMaxDim, gemm::kNumConfigs - 1, 1 << 20, 3, 1};
        for (int i = 0; i < 8 && rc == GEMM_OK; ++i)
            if (!parse_field(&s, lo[i], hi[i], &v[i])) rc = GEMM_ERR_INVALID_VALUE;
        while (rc == GEMM_OK && (*s == ' ' || *s == '\t' || *s == '\r' || *s == '\n')) ++s;
        if (rc == GEMM_OK && *s != '\0') rc = GEMM_ERR_INVALID_VALUE;            // trailing text
        if (rc == GEMM_OK)
            out->push_back({Shape{int32_t(v[0]), v[1], v[2], v[3], int32_t(v[7])},
                            LoadedPlan{int32_t(v[4]), int32_t(v[5]), int32_t(v[6])}});
    }
    if (ferror(f)) rc = GEMM_ERR_INVALID_VALUE;
    fclose(f);
    return rc;
}

// Adds every plan of the file to the loaded ones (a later line for the same shape wins).
int load_plan_file(const char *path) {
    std::vector<std::pair<Shape, LoadedPlan>> plans;
    const int rc = read_plan_file(path, &plans);
    if (rc != GEMM_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    for (const auto &kv : plans) g_loaded[kv.first] = kv.second;
    g_cache.clear();
    return GEMM_OK;
}

// GEMM_MI355X_PLANS names a plan file to load before the first plan is chosen.
void load_env_plans() {
    const char *path = getenv("GEMM_MI355X_PLANS");
    if (path == nullptr || *path == '\0') return;
    if (load_plan_file(path) != GEMM_OK)
        fprintf(stderr, "gemm_mi355x: GEMM_MI355X_PLANS=%s not loaded (unreadable file or malformed line)\n", path);
}

bool overlaps(uintptr_t a0, uint64_t alen, uintptr_t b0, uint64_t blen) {
    if (alen == 0 || blen == 0) return false;
    return a0 < b0 + blen && b0 < a0 + alen;
}

// Bytes spanned by a row-major rows x cols matrix with row stride ld.
uint64_t span_bytes(int64_t rows, int64_t cols, int64_t ld, int64_t esize) {
    if (rows <= 0 || cols <= 0) return 0;
    return uint64_t((rows - 1) * ld + cols) * uint64_t(esize);
}

// c_esize: bytes per element of C (4 for the int32 / fp32 outputs, 1 or 2 for the
// reduced-precision ones).
int validate(const Problem &p, const void *A, const void *B, const void *C, int64_t c_esize = 4) {
    if (p.M < 0 || p.N < 0 || p.K < 0) return GEMM_ERR_INVALID_VALUE;
    const int64_t e = gemm::elem_bytes(p.dtype);
    const bool has_a = p.M > 0 && p.K > 0, has_b = p.K > 0 && p.N > 0, has_c = p.M > 0 && p.N > 0;
    // B is K x N row-major (rows of N), or stored column-major as N x K (rows of K).
    const int64_t b_rows = p.trans_b ? p.N : p.K, b_cols = p.trans_b ? p.K : p.N;
    if (has_a && (A == nullptr || p.lda < p.K)) return GEMM_ERR_INVALID_VALUE;
    if (has_b && (B == nullptr || p.ldb < b_cols)) return GEMM_ERR_INVALID_VALUE;
    if (has_c && (C == nullptr || p.ldc < p.N)) return GEMM_ERR_INVALID_VALUE;
    // Natural alignment of the element types (a misaligned int32*/float*/bf16* is not a valid pointer).
    if (has_a && (uintptr_t(A) % uintptr_t(e)) != 0) return GEMM_ERR_INVALID_VALUE;
    if (has_b && (uintptr_t(B) % uintptr_t(e)) != 0) return GEMM_ERR_INVALID_VALUE;
    if (has_c && (uintptr_t(C) % uintptr_t(c_esize)) != 0) return GEMM_ERR_INVALID_VALUE;
    // Stride products must not overflow 64-bit byte offsets.
    const int64_t lim = int64_t(1) << 55;
    if (p.M > lim || p.N > lim || p.K > lim || (has_a && p.lda > lim / (p.M > 0 ? p.M : 1)) ||
        (has_b && p.ldb > lim / (b_rows > 0 ? b_rows : 1)) || (has_c && p.ldc > lim / (p.M > 0 ? p.M : 1)))
        return GEMM_ERR_INVALID_VALUE;
    const uint64_t clen = span_bytes(p.M, p.N, p.ldc, c_esize);
    if (has_c && has_a && overlaps(uintptr_t(C), clen, uintptr_t(A), span_bytes(p.M, p.K, p.lda, e)))
        return GEMM_ERR_INVALID_VALUE;
    if (has_c && has_b && overlaps(uintptr_t(C), clen, uintptr_t(B), span_bytes(b_rows, b_cols, p.ldb, e)))
        return GEMM_ERR_INVALID_VALUE;
    return GEMM_OK;
}

// The plan for a call, and where it came from (GEMM_PLAN_FROM_*) if `source` is given.
int plan_for(const Problem &p, Plan *out, int32_t *source = nullptr) {
    std::call_once(g_env_once, load_env_plans);
    Override ov;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        ov = g_override[p.dtype];
    }
    const bool forced = ov.family >= 0 || ov.config >= 0 || ov.split > 0 || ov.reduce >= 0;
    if (!forced) {
        const Key key{p.dtype, p.M, p.N, p.K, gemm::vector_loads_ok(p), p.trans_b};
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_cache.find(key);
        if (it != g_cache.end()) {
            *out = it->second.plan;
            if (source) *source = it->second.source;
            return GEMM_OK;
        }
    }
    Plan pl;
    bool loaded = false;
    if (!forced) {
        LoadedPlan lp{};
        {
            std::lock_guard<std::mutex> lk(g_mu);
            auto it = g_loaded.find(Shape{p.dtype, p.M, p.N, p.K, p.trans_b});
            loaded = it != g_loaded.end();
            if (loaded) lp = it->second;
        }
        // A loaded plan whose configuration cannot run this call (alignment) is skipped.
        loaded = loaded && gemm::config_applicable(p, lp.config);
        if (loaded) pl = gemm::evaluate(p, lp.config, lp.split, gemm::Chip(), lp.reduce);
    }
    if (!loaded && !gemm::select_plan(p, &pl, ov.family, ov.config, ov.split, gemm::Chip(), ov.reduce))
        return GEMM_ERR_UNSUPPORTED;
    // select_plan consults the compiled table, then the nearest-M neighbours, then the model.
    int32_t cfg, split, reduce;
    const int32_t src = forced ? GEMM_PLAN_FROM_FORCED
                      : loaded ? GEMM_PLAN_FROM_FILE
                      : gemm::tuned_plan(p, &cfg, &split, &reduce) ? GEMM_PLAN_FROM_TABLE
                      : gemm::neighbour_plan(p, &cfg, &split, &reduce) ? GEMM_PLAN_FROM_NEIGHBOUR
                      : GEMM_PLAN_FROM_MODEL;
    if (!forced) {
        const Key key{p.dtype, p.M, p.N, p.K, gemm::vector_loads_ok(p), p.trans_b};
        std::lock_guard<std::mutex> lk(g_mu);
        if (g_cache.size() > 4096) g_cache.clear();
        g_cache.emplace(key, CachedPlan{pl, src});
    }
    *out = pl;
    if (source) *source = src;
    return GEMM_OK;
}

int run(int32_t dtype, int32_t trans_b, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
        const void *B, int64_t ldb, void *C, int64_t ldc, void *stream,
        int32_t epilogue = gemm::EPI_NONE, int32_t shift = 0, bool static_scratch = false) {
    Problem p{dtype, M, N, K, lda, ldb, ldc, uintptr_t(A), uintptr_t(B), uintptr_t(C), trans_b};
    const int64_t c_esize = epilogue == gemm::EPI_I8 ? 1 : (epilogue == gemm::EPI_NONE ? 4 : 2);
    if (shift < 0 || shift > 31) return GEMM_ERR_INVALID_VALUE;
    int rc = validate(p, A, B, C, c_esize);
    if (rc != GEMM_OK) return rc;
    if (M == 0 || N == 0) return GEMM_OK;
    Plan pl;
    rc = plan_for(p, &pl);
    if (rc != GEMM_OK) return rc;

    gemm::KernelArgs a{};
    a.dtype = dtype;
    a.A = A;
    a.B = B;
    a.C = C;
    a.workspace = nullptr;
    a.M = M; a.N = N; a.K = K;
    a.lda = K > 0 ? lda : 0;
    a.ldb = K > 0 ? ldb : 0;
    a.ldc = ldc;
    a.k_chunk = pl.k_chunk;
    a.split_k = pl.split_k;
    a.tiles_m = int32_t(pl.tiles_m);
    a.tiles_n = int32_t(pl.tiles_n);
    a.group_m = 4;
    a.reduce_in_kernel = pl.reduce_in_kernel;
    // The atomic reductions add int32 partials into C: narrowed outputs take the separate one.
    if ((a.reduce_in_kernel == gemm::REDUCE_ATOMIC || a.reduce_in_kernel == gemm::REDUCE_ATOMIC_FLAG) &&
        epilogue != gemm::EPI_NONE)
        a.reduce_in_kernel = gemm::REDUCE_SEPARATE;
    a.b_trans = trans_b;
    a.epilogue = epilogue;
    a.shift = shift;
    if (pl.grid > 0x7fffffff || pl.tiles_m > 0x7fffffff || pl.tiles_n > 0x7fffffff)
        return GEMM_ERR_UNSUPPORTED;
    const int lr = gemm::launch_gemm(a, pl.config, pl.grid, stream, static_scratch);
    if (lr == gemm::LAUNCH_NO_MEMORY) return GEMM_ERR_NO_MEMORY;
    if (lr == gemm::LAUNCH_SCRATCH_LIMIT) return GEMM_ERR_SCRATCH_LIMIT;
    if (lr != gemm::LAUNCH_OK) return GEMM_ERR_HIP;
    return GEMM_OK;
}

}  // namespace

extern "C" {

int gemm_i8_i32(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *B,
                int64_t ldb, int32_t *C, int64_t ldc, void *stream) {
    return run(gemm::DT_I8, 0, M, N, K, A, lda, B, ldb, C, ldc, stream);
}

int gemm_bf16_f32(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda, const uint16_t *B,
                  int64_t ldb, float *C, int64_t ldc, void *stream) {
    return run(gemm::DT_BF16, 0, M, N, K, A, lda, B, ldb, C, ldc, stream);
}

int gemm_bf16_f32_noalloc(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda, const uint16_t *B,
                          int64_t ldb, float *C, int64_t ldc, void *stream) {
    return run(gemm::DT_BF16, 0, M, N, K, A, lda, B, ldb, C, ldc, stream, gemm::EPI_NONE, 0, true);
}

int gemm_i8_i32_bt(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *Bt,
                   int64_t ldbt, int32_t *C, int64_t ldc, void *stream) {
    return run(gemm::DT_I8, 1, M, N, K, A, lda, Bt, ldbt, C, ldc, stream);
}

int gemm_bf16_f32_bt(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda, const uint16_t *Bt,
                     int64_t ldbt, float *C, int64_t ldc, void *stream) {
    return run(gemm::DT_BF16, 1, M, N, K, A, lda, Bt, ldbt, C, ldc, stream);
}

int gemm_i8_i8(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *B,
               int64_t ldb, int8_t *C, int64_t ldc, int shift, void *stream) {
    return run(gemm::DT_I8, 0, M, N, K, A, lda, B, ldb, C, ldc, stream, gemm::EPI_I8, shift);
}

int gemm_i8_i16(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *B,
                int64_t ldb, int16_t *C, int64_t ldc, int shift, void *stream) {
    return run(gemm::DT_I8, 0, M, N, K, A, lda, B, ldb, C, ldc, stream, gemm::EPI_I16, shift);
}

int gemm_bf16_bf16(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda, const uint16_t *B,
                   int64_t ldb, uint16_t *C, int64_t ldc, void *stream) {
    return run(gemm::DT_BF16, 0, M, N, K, A, lda, B, ldb, C, ldc, stream, gemm::EPI_BF16, 0);
}

int gemm_i8_i8_bt(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *Bt,
                  int64_t ldbt, int8_t *C, int64_t ldc, int shift, void *stream) {
    return run(gemm::DT_I8, 1, M, N, K, A, lda, Bt, ldbt, C, ldc, stream, gemm::EPI_I8, shift);
}

int gemm_i8_i16_bt(int64_t M, int64_t N, int64_t K, const int8_t *A, int64_t lda, const int8_t *Bt,
                   int64_t ldbt, int16_t *C, int64_t ldc, int shift, void *stream) {
    return run(gemm::DT_I8, 1, M, N, K, A, lda, Bt, ldbt, C, ldc, stream, gemm::EPI_I16, shift);
}

int gemm_bf16_bf16_bt(int64_t M, int64_t N, int64_t K, const uint16_t *A, int64_t lda, const uint16_t *Bt,
                      int64_t ldbt, uint16_t *C, int64_t ldc, void *stream) {
    return run(gemm::DT_BF16, 1, M, N, K, A, lda, Bt, ldbt, C, ldc, stream, gemm::EPI_BF16, 0);
}

static int plan_impl(int dtype, int32_t trans_b, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb,
                     int64_t ldc, uintptr_t a_addr, uintptr_t b_addr, uintptr_t c_addr, gemm_plan_info *out) {
    if (out == nullptr || (dtype != GEMM_DTYPE_I8_I32 && dtype != GEMM_DTYPE_BF16_F32))
        return GEMM_ERR_INVALID_VALUE;
    Problem p{dtype, M, N, K, lda, ldb, ldc, a_addr, b_addr, c_addr, trans_b};
    int rc = validate(p, reinterpret_cast<const void *>(a_addr), reinterpret_cast<const void *>(b_addr),
                      reinterpret_cast<const void *>(c_addr));
    if (rc != GEMM_OK) return rc;
    memset(out, 0, sizeof(*out));
    if (M == 0 || N == 0) {
        out->kernel = -1;
        out->config = -1;
        strncpy(out->name, "noop", sizeof(out->name) - 1);
        return GEMM_OK;
    }
    Plan pl;
    int32_t source = GEMM_PLAN_FROM_MODEL;
    rc = plan_for(p, &pl, &source);
    if (rc != GEMM_OK) return rc;
    const gemm::TileConfig &c = gemm::kConfigs[pl.config];
    out->kernel = c.family;
    out->config = pl.config;
    out->bm = c.bm;
    out->bn = c.bn;
    out->bk = gemm::stage_k_elems(dtype);
    out->waves = c.wm * c.wn;
    const bool mfma = c.family != gemm::FAM_GEMV;      // the matrix-vector kernels use the vector ALUs
    out->mfma_m = mfma ? 32 : 0;
    out->mfma_n = mfma ? 32 : 0;
    out->mfma_k = mfma ? (dtype == GEMM_DTYPE_I8_I32 ? 32 : 16) : 0;
    out->split_k = pl.split_k;
    out->reduce_in_kernel = pl.split_k > 1 ? pl.reduce_in_kernel : 0;
    out->k_chunk = pl.k_chunk;
    out->grid = pl.grid;
    out->lds_bytes = gemm::lds_bytes(c);
    out->workspace_bytes = pl.workspace_bytes;
    out->model_traffic_bytes = pl.traffic_bytes;
    out->model_t_comp_us = pl.t_comp_us;
    out->model_t_mem_us = pl.t_mem_us;
    out->source = source;
    strncpy(out->name, c.name, sizeof(out->name) - 1);
    return GEMM_OK;
}

int gemm_plan(int dtype, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc,
              uintptr_t a_addr, uintptr_t b_addr, uintptr_t c_addr, gemm_plan_info *out) {
    return plan_impl(dtype, 0, M, N, K, lda, ldb, ldc, a_addr, b_addr, c_addr, out);
}

int gemm_plan_bt(int dtype, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldbt, int64_t ldc,
                 uintptr_t a_addr, uintptr_t bt_addr, uintptr_t c_addr, gemm_plan_info *out) {
    return plan_impl(dtype, 1, M, N, K, lda, ldbt, ldc, a_addr, bt_addr, c_addr, out);
}

int gemm_force_plan(int dtype, int kernel, int config, int split_k) {
    if (dtype != GEMM_DTYPE_I8_I32 && dtype != GEMM_DTYPE_BF16_F32) return GEMM_ERR_INVALID_VALUE;
    if (split_k < 0 || config < -1 || config >= gemm::kNumConfigs) return GEMM_ERR_INVALID_VALUE;
    if (kernel < GEMM_KERNEL_AUTO || kernel > GEMM_KERNEL_GEMV) return GEMM_ERR_INVALID_VALUE;
    if (config >= 0 && kernel >= 0 && gemm::kConfigs[config].family != kernel) return GEMM_ERR_INVALID_VALUE;
    std::lock_guard<std::mutex> lk(g_mu);
    Override &o = g_override[dtype];
    if (kernel == GEMM_KERNEL_AUTO && config < 0) {
        o.family = -1;
        o.config = -1;
        o.split = split_k;
    } else {
        o.family = kernel;
        o.config = config;
        o.split = split_k;
    }
    return GEMM_OK;
}

int gemm_force_reduce(int dtype, int mode) {
    if (dtype != GEMM_DTYPE_I8_I32 && dtype != GEMM_DTYPE_BF16_F32) return GEMM_ERR_INVALID_VALUE;
    if (mode < -1 || mode > 3) return GEMM_ERR_INVALID_VALUE;
    std::lock_guard<std::mutex> lk(g_mu);
    g_override[dtype].reduce = mode;
    return GEMM_OK;
}

int gemm_load_plans(const char *path) {
    std::call_once(g_env_once, load_env_plans);
    return load_plan_file(path);
}

int gemm_clear_plans(void) {
    std::call_once(g_env_once, load_env_plans);
    std::lock_guard<std::mutex> lk(g_mu);
    g_loaded.clear();
    g_cache.clear();
    return GEMM_OK;
}

int gemm_release_workspace(void) {
    return gemm::release_workspaces() == gemm::LAUNCH_OK ? GEMM_OK : GEMM_ERR_HIP;
}

const char *gemm_status_string(int status) {
    switch (status) {
        case GEMM_OK: return "GEMM_OK: success";
        case GEMM_ERR_INVALID_VALUE: return "GEMM_ERR_INVALID_VALUE: invalid argument";
        case GEMM_ERR_UNSUPPORTED: return "GEMM_ERR_UNSUPPORTED: no kernel can run this plan";
        case GEMM_ERR_HIP: return "GEMM_ERR_HIP: HIP launch or runtime error";
        case GEMM_ERR_NO_MEMORY: return "GEMM_ERR_NO_MEMORY: split-K workspace allocation failed";
        case GEMM_ERR_SCRATCH_LIMIT:
            return "GEMM_ERR_SCRATCH_LIMIT: the plan's split-K partials exceed the fixed scratch of "
                   "gemm_bf16_f32_noalloc";
        default: return "unknown gemm status";
    }
}

const char *gemm_version(void) { return "gemm_mi355x 0.1 (gfx950)"; }

}  // extern "C"
