// som_api.cpp -- host side of the C ABI declared in include/som.h: argument checks,
// workspace carving, launches on the caller's stream, error text.

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cmath>
#include <cstring>

#include "../../include/som.h"
#include "som_internal.h"

namespace {

thread_local char g_err[512] = "";

som_status fail(som_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

som_status hip_fail(hipError_t e, const char *what)
{
    return fail(SOM_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

som_status ok()
{
    g_err[0] = '\0';
    return SOM_OK;
}

struct Opts {
    int ta;      // samples per tile
    bool order;  // reorder samples by their least frequent feature
};

// Options from the optional config.
som_status parse(const som_bmu_config *cfg, Opts *o)
{
    o->ta = som::kDefaultTileSamples;
    o->order = true;
    if (!cfg) return SOM_OK;
    for (int r : cfg->reserved)
        if (r != 0) return fail(SOM_ERR_INVALID_ARG, "som_bmu_config.reserved must be zero");
    if (cfg->tile_samples != 0) {
        if (!som::valid_tile(cfg->tile_samples))
            return fail(SOM_ERR_INVALID_ARG, "tile_samples must be 0, 8, 16 or 32 (got %d)", (int)cfg->tile_samples);
        o->ta = cfg->tile_samples;
    }
    if (cfg->keep_order != 0 && cfg->keep_order != 1)
        return fail(SOM_ERR_INVALID_ARG, "keep_order must be 0 or 1 (got %d)", (int)cfg->keep_order);
    o->order = cfg->keep_order == 0;
    return SOM_OK;
}

som_status check_dims(int64_t N, int64_t M, int64_t V, int64_t nnz)
{
    if (N < 0 || N >= INT32_MAX) return fail(SOM_ERR_INVALID_ARG, "N must be in [0, 2^31-1) (got %lld)", (long long)N);
    if (M < 1 || M > SOM_MAX_NEURONS)
        return fail(SOM_ERR_INVALID_ARG, "M must be in [1, %d] (got %lld)", SOM_MAX_NEURONS, (long long)M);
    if (V < 1 || V >= INT32_MAX) return fail(SOM_ERR_INVALID_ARG, "V must be in [1, 2^31-1) (got %lld)", (long long)V);
    if (nnz < 0 || nnz > INT32_MAX)
        return fail(SOM_ERR_INVALID_ARG, "nnz must be in [0, 2^31-1] (got %lld)", (long long)nnz);
    return SOM_OK;
}

bool dims_ok(int64_t N, int64_t M, int64_t V, int64_t nnz)
{
    return !(N < 0 || N >= INT32_MAX || M < 1 || M > SOM_MAX_NEURONS || V < 1 || V >= INT32_MAX || nnz < 0 ||
             nnz > INT32_MAX);
}

// Which workspace layout a call works on. Binary rows: single-best, or two-best (a
// superset). Real-valued rows: always the two-best layout plus the value sections.
struct Kind {
    bool top2;  // produce the two best units
    bool real;  // real-valued rows
    bool layout_top2() const { return top2 || real; }
};

struct Carved {
    uint2 *plan;
    int2 *tiles;
    som::SweepOut out;
    uint32_t *flags;
    som::OrderBuffers ob;
    float *vals;
    double *xsq;
};

som_status carve(void *ws, size_t bytes, int64_t N, int64_t M, int64_t V, int64_t nnz, const Opts &o, const Kind &k,
                 Carved *c)
{
    if (!ws) return fail(SOM_ERR_WORKSPACE, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(ws) & 255) return fail(SOM_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    const som::Layout L = som::layout_for(N, M, V, nnz, o.ta, o.order, k.layout_top2(), k.real);
    if (bytes < L.total)
        return fail(SOM_ERR_WORKSPACE, "workspace holds %zu bytes, the search needs %zu", bytes, L.total);
    char *b = static_cast<char *>(ws);
    c->plan = reinterpret_cast<uint2 *>(b + L.plan);
    c->tiles = reinterpret_cast<int2 *>(b + L.tiles);
    c->out.keys = reinterpret_cast<unsigned long long *>(b + L.keys);
    c->out.dots = reinterpret_cast<float *>(b + L.dots);
    c->out.keys2 = k.layout_top2() ? reinterpret_cast<unsigned long long *>(b + L.keys2) : nullptr;
    c->out.dots2 = k.layout_top2() ? reinterpret_cast<float *>(b + L.dots2) : nullptr;
    c->flags = reinterpret_cast<uint32_t *>(b + L.flags);
    c->ob.freq = reinterpret_cast<uint32_t *>(b + L.freq);
    c->ob.bucket = reinterpret_cast<unsigned long long *>(b + L.bucket);
    c->ob.skey = reinterpret_cast<int32_t *>(b + L.skey);
    c->ob.rank = reinterpret_cast<unsigned long long *>(b + L.rank);
    c->ob.inv = reinterpret_cast<int32_t *>(b + L.inv);
    c->ob.res = reinterpret_cast<som::Staged *>(b + L.res);
    c->ob.res2 = k.layout_top2() ? reinterpret_cast<som::Staged *>(b + L.res2) : nullptr;
    c->ob.pos = reinterpret_cast<int32_t *>(b + L.pos);
    c->vals = k.real ? reinterpret_cast<float *>(b + L.vals) : nullptr;
    c->xsq = k.real ? reinterpret_cast<double *>(b + L.xsq) : nullptr;
    return SOM_OK;
}

// Common prologue of the phases: options, N == 0 (a no-op), workspace.
som_status setup(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config, void *workspace,
                 size_t workspace_bytes, const Kind &k, Opts *o, Carved *c, bool *noop)
{
    som_status st = parse(config, o);
    if (st != SOM_OK) return st;
    if (k.real && o->ta != 8)
        return fail(SOM_ERR_INVALID_ARG, "real-valued rows use tiles of 8 samples (tile_samples 0 or 8)");
    *noop = N == 0;
    if (*noop) return SOM_OK;
    return carve(workspace, workspace_bytes, N, M, V, nnz, *o, k, c);
}

size_t workspace_for(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config, const Kind &k)
{
    if (!dims_ok(N, M, V, nnz)) return 0;
    Opts o;
    if (parse(config, &o) != SOM_OK) return 0;
    if (k.real && o.ta != 8) return 0;
    return som::layout_for(N, M, V, nnz, o.ta, o.order, k.layout_top2(), k.real).total;
}

// A codebook: fp32, or IEEE binary16 bit patterns.
struct Book {
    const void *p;
    bool f16;
};

som_status check_book(const Book &b, const char *who)
{
    if (reinterpret_cast<uintptr_t>(b.p) & (b.f16 ? 1 : 3))
        return fail(SOM_ERR_INVALID_ARG, "%s: W must be %d-byte aligned", who, b.f16 ? 2 : 4);
    return SOM_OK;
}

som_status norms_impl(const Book &b, int64_t V, int64_t M, double *norms, void *stream, const char *who)
{
    if (!b.p || !norms) return fail(SOM_ERR_INVALID_ARG, "%s: null pointer", who);
    if (M < 1 || M > SOM_MAX_NEURONS || V < 1 || V >= INT32_MAX)
        return fail(SOM_ERR_INVALID_ARG, "%s: need 1 <= M <= %d and 1 <= V < 2^31-1", who, SOM_MAX_NEURONS);
    som_status st = check_book(b, who);
    if (st != SOM_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = b.f16 ? som::launch_norms_f16(static_cast<const uint16_t *>(b.p), V, M, norms, s)
                         : som::launch_norms(static_cast<const float *>(b.p), V, M, norms, s);
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

som_status plan_impl(const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N, int64_t nnz,
                     int64_t V, int64_t M, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                     void *stream, const Kind &k, const char *who)
{
    Opts o;
    Carved c;
    bool noop;
    som_status st = check_dims(N, M, V, nnz);
    if (st != SOM_OK) return st;
    if (N > 0 && (!row_ptr || (nnz > 0 && (!col_idx || (k.real && !values)))))
        return fail(SOM_ERR_INVALID_ARG, "%s: null CSR pointer", who);
    if ((st = setup(N, M, V, nnz, config, workspace, workspace_bytes, k, &o, &c, &noop)) != SOM_OK) return st;
    if (noop) return ok();
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = som::launch_clear_flags(c.flags, s);
    if (e != hipSuccess) return hip_fail(e, who);
    e = som::launch_check_rows(row_ptr, N, nnz, c.flags, s);
    if (e != hipSuccess) return hip_fail(e, who);
    if (o.order) {
        e = som::launch_order(row_ptr, col_idx, N, nnz, V, c.ob, c.flags, s);
        if (e != hipSuccess) return hip_fail(e, who);
    }
    e = som::launch_plan(o.ta, row_ptr, col_idx, k.real ? values : nullptr, N, nnz, V, o.order ? &c.ob : nullptr,
                         c.plan, c.tiles, c.vals, c.xsq, c.flags, s);
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

som_status sweep_impl(const Book &b, const Kind &k, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                      void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream,
                      const char *who)
{
    Opts o;
    Carved c;
    bool noop;
    som_status st = check_dims(N, M, V, nnz);
    if (st != SOM_OK) return st;
    if (N > 0 && (!b.p || !norms)) return fail(SOM_ERR_INVALID_ARG, "%s: null pointer", who);
    if ((st = check_book(b, who)) != SOM_OK) return st;
    if ((st = setup(N, M, V, nnz, config, workspace, workspace_bytes, k, &o, &c, &noop)) != SOM_OK) return st;
    if (noop) return ok();
    som::SweepOut out = c.out;
    if (!k.top2) out.keys2 = nullptr, out.dots2 = nullptr;
    hipError_t e = som::launch_sweep(o.ta, b.f16, k.top2, b.p, norms, M, N, V, nnz, c.plan, c.tiles, c.vals, out,
                                     static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

som_status finalize_impl(const Kind &k, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N,
                         int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2, void *workspace,
                         size_t workspace_bytes, const som_bmu_config *config, void *stream, const char *who)
{
    Opts o;
    Carved c;
    bool noop;
    som_status st = check_dims(N, M, V, nnz);
    if (st != SOM_OK) return st;
    if (N > 0 && (!norms || !row_ptr || !bmu || !dist || (k.top2 && (!bmu2 || !dist2))))
        return fail(SOM_ERR_INVALID_ARG, "%s: null pointer", who);
    if ((st = setup(N, M, V, nnz, config, workspace, workspace_bytes, k, &o, &c, &noop)) != SOM_OK) return st;
    if (noop) return ok();
    hipError_t e = som::launch_finalize(o.ta, norms, M, row_ptr, N, nnz, o.order ? &c.ob : nullptr, c.xsq, c.out, bmu, dist,
                                        k.top2 ? bmu2 : nullptr, k.top2 ? dist2 : nullptr,
                                        static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

som_status search_impl(const Book &b, const Kind &k, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                       const int32_t *col_idx, const float *values, int64_t N, int64_t nnz, int32_t *bmu,
                       double *dist, int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                       const som_bmu_config *config, void *stream, const char *who)
{
    Opts o;
    Carved c;
    bool noop;
    som_status st = check_dims(N, M, V, nnz);
    if (st != SOM_OK) return st;
    if (N > 0 && (!b.p || !norms || !row_ptr || (nnz > 0 && (!col_idx || (k.real && !values))) || !bmu || !dist ||
                  (k.top2 && (!bmu2 || !dist2))))
        return fail(SOM_ERR_INVALID_ARG, "%s: null pointer", who);
    if ((st = check_book(b, who)) != SOM_OK) return st;
    if ((st = setup(N, M, V, nnz, config, workspace, workspace_bytes, k, &o, &c, &noop)) != SOM_OK) return st;
    if (noop) return ok();
    if ((st = plan_impl(row_ptr, col_idx, values, N, nnz, V, M, workspace, workspace_bytes, config, stream, k, who)) !=
        SOM_OK)
        return st;
    if ((st = sweep_impl(b, k, norms, V, M, N, nnz, workspace, workspace_bytes, config, stream, who)) != SOM_OK)
        return st;
    return finalize_impl(k, norms, V, M, row_ptr, N, nnz, bmu, dist, bmu2, dist2, workspace, workspace_bytes, config,
                         stream, who);
}

constexpr Kind kOne{false, false}, kTwo{true, false};

Kind real_kind(const int32_t *bmu2, const double *dist2) { return Kind{bmu2 != nullptr || dist2 != nullptr, true}; }

}  // namespace

som_status som::set_error(som_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

extern "C" {

size_t som_bmu_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config)
{
    return workspace_for(N, M, V, nnz, config, kOne);
}

size_t som_bmu2_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config)
{
    return workspace_for(N, M, V, nnz, config, kTwo);
}

size_t som_bmu_sf_workspace_bytes(int64_t N, int64_t M, int64_t V, int64_t nnz, const som_bmu_config *config)
{
    return workspace_for(N, M, V, nnz, config, Kind{true, true});
}

som_status som_codebook_norms(const float *W, int64_t V, int64_t M, double *norms, void *stream)
{
    return norms_impl(Book{W, false}, V, M, norms, stream, "som_codebook_norms");
}

som_status som_codebook_norms_f16(const uint16_t *W, int64_t V, int64_t M, double *norms, void *stream)
{
    return norms_impl(Book{W, true}, V, M, norms, stream, "som_codebook_norms_f16");
}

som_status som_bmu_plan(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t nnz, int64_t V, int64_t M,
                        void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return plan_impl(row_ptr, col_idx, nullptr, N, nnz, V, M, workspace, workspace_bytes, config, stream, kOne,
                     "som_bmu_plan");
}

som_status som_bmu_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                         void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return sweep_impl(Book{W, false}, kOne, norms, V, M, N, nnz, workspace, workspace_bytes, config, stream,
                      "som_bmu_sweep");
}

som_status som_bmu_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                             void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return sweep_impl(Book{W, true}, kOne, norms, V, M, N, nnz, workspace, workspace_bytes, config, stream,
                      "som_bmu_sweep_f16");
}

som_status som_bmu_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N, int64_t nnz,
                            int32_t *bmu, double *dist, void *workspace, size_t workspace_bytes,
                            const som_bmu_config *config, void *stream)
{
    return finalize_impl(kOne, norms, V, M, row_ptr, N, nnz, bmu, dist, nullptr, nullptr, workspace, workspace_bytes,
                         config, stream, "som_bmu_finalize");
}

som_status som_bmu_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                          const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                          void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return search_impl(Book{W, false}, kOne, norms, V, M, row_ptr, col_idx, nullptr, N, nnz, bmu, dist, nullptr,
                       nullptr, workspace, workspace_bytes, config, stream, "som_bmu_search");
}

som_status som_bmu_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                              const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                              void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return search_impl(Book{W, true}, kOne, norms, V, M, row_ptr, col_idx, nullptr, N, nnz, bmu, dist, nullptr,
                       nullptr, workspace, workspace_bytes, config, stream, "som_bmu_search_f16");
}

som_status som_bmu2_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                          void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return sweep_impl(Book{W, false}, kTwo, norms, V, M, N, nnz, workspace, workspace_bytes, config, stream,
                      "som_bmu2_sweep");
}

som_status som_bmu2_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                              void *workspace, size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return sweep_impl(Book{W, true}, kTwo, norms, V, M, N, nnz, workspace, workspace_bytes, config, stream,
                      "som_bmu2_sweep_f16");
}

som_status som_bmu2_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N,
                             int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2, void *workspace,
                             size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return finalize_impl(kTwo, norms, V, M, row_ptr, N, nnz, bmu, dist, bmu2, dist2, workspace, workspace_bytes,
                         config, stream, "som_bmu2_finalize");
}

som_status som_bmu2_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                           const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2,
                           double *dist2, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                           void *stream)
{
    return search_impl(Book{W, false}, kTwo, norms, V, M, row_ptr, col_idx, nullptr, N, nnz, bmu, dist, bmu2, dist2,
                       workspace, workspace_bytes, config, stream, "som_bmu2_search");
}

som_status som_bmu2_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                               const int32_t *col_idx, int64_t N, int64_t nnz, int32_t *bmu, double *dist,
                               int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                               const som_bmu_config *config, void *stream)
{
    return search_impl(Book{W, true}, kTwo, norms, V, M, row_ptr, col_idx, nullptr, N, nnz, bmu, dist, bmu2, dist2,
                       workspace, workspace_bytes, config, stream, "som_bmu2_search_f16");
}

som_status som_bmu_sf_plan(const int32_t *row_ptr, const int32_t *col_idx, const float *values, int64_t N,
                           int64_t nnz, int64_t V, int64_t M, void *workspace, size_t workspace_bytes,
                           const som_bmu_config *config, void *stream)
{
    return plan_impl(row_ptr, col_idx, values, N, nnz, V, M, workspace, workspace_bytes, config, stream,
                     Kind{true, true}, "som_bmu_sf_plan");
}

som_status som_bmu_sf_sweep(const float *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                            int32_t two_best, void *workspace, size_t workspace_bytes, const som_bmu_config *config,
                            void *stream)
{
    return sweep_impl(Book{W, false}, Kind{two_best != 0, true}, norms, V, M, N, nnz, workspace, workspace_bytes,
                      config, stream, "som_bmu_sf_sweep");
}

som_status som_bmu_sf_sweep_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, int64_t N, int64_t nnz,
                                int32_t two_best, void *workspace, size_t workspace_bytes,
                                const som_bmu_config *config, void *stream)
{
    return sweep_impl(Book{W, true}, Kind{two_best != 0, true}, norms, V, M, N, nnz, workspace, workspace_bytes,
                      config, stream, "som_bmu_sf_sweep_f16");
}

som_status som_bmu_sf_finalize(const double *norms, int64_t V, int64_t M, const int32_t *row_ptr, int64_t N,
                               int64_t nnz, int32_t *bmu, double *dist, int32_t *bmu2, double *dist2, void *workspace,
                               size_t workspace_bytes, const som_bmu_config *config, void *stream)
{
    return finalize_impl(real_kind(bmu2, dist2), norms, V, M, row_ptr, N, nnz, bmu, dist, bmu2, dist2, workspace,
                         workspace_bytes, config, stream, "som_bmu_sf_finalize");
}

som_status som_bmu_sf_search(const float *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                             const int32_t *col_idx, const float *values, int64_t N, int64_t nnz, int32_t *bmu,
                             double *dist, int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                             const som_bmu_config *config, void *stream)
{
    return search_impl(Book{W, false}, real_kind(bmu2, dist2), norms, V, M, row_ptr, col_idx, values, N, nnz, bmu,
                       dist, bmu2, dist2, workspace, workspace_bytes, config, stream, "som_bmu_sf_search");
}

som_status som_bmu_sf_search_f16(const uint16_t *W, const double *norms, int64_t V, int64_t M, const int32_t *row_ptr,
                                 const int32_t *col_idx, const float *values, int64_t N, int64_t nnz, int32_t *bmu,
                                 double *dist, int32_t *bmu2, double *dist2, void *workspace, size_t workspace_bytes,
                                 const som_bmu_config *config, void *stream)
{
    return search_impl(Book{W, true}, real_kind(bmu2, dist2), norms, V, M, row_ptr, col_idx, values, N, nnz, bmu,
                       dist, bmu2, dist2, workspace, workspace_bytes, config, stream, "som_bmu_sf_search_f16");
}

som_status som_bmu_input_flags(const void *workspace, size_t workspace_bytes, int64_t N, int64_t M, int64_t V,
                               int64_t nnz, const som_bmu_config *config, uint32_t *flags, void *stream)
{
    Opts o;
    Carved c;
    bool noop;
    som_status st = check_dims(N, M, V, nnz);
    if (st != SOM_OK) return st;
    if (!flags) return fail(SOM_ERR_INVALID_ARG, "som_bmu_input_flags: flags is NULL");
    *flags = 0;
    // the flags lead every layout; the single-best one is a prefix of all others
    if ((st = setup(N, M, V, nnz, config, const_cast<void *>(workspace), workspace_bytes, kOne, &o, &c, &noop)) !=
        SOM_OK)
        return st;
    if (noop) return ok();
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "som_bmu_input_flags: stream synchronize");
    e = hipMemcpy(flags, c.flags, sizeof(uint32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "som_bmu_input_flags: copy");
    return ok();
}

size_t som_update_workspace_bytes(int64_t V, int64_t E, int64_t N, int64_t chunk_features)
{
    if (V < 1 || V >= INT32_MAX || E < 1 || E * E > SOM_MAX_NEURONS || N < 0 || N >= INT32_MAX || chunk_features < 0)
        return 0;
    const int64_t chunk = chunk_features == 0 || chunk_features > V ? V : chunk_features;
    return som::update_layout(E * E, N, chunk).total;
}

static som_status update_impl(const Book &b, void *W, int64_t V, int64_t E, const int32_t *row_ptr,
                              const int32_t *col_idx, int64_t N, int64_t nnz, const int32_t *bmu, int32_t radius,
                              int64_t chunk_features, void *workspace, size_t workspace_bytes, void *stream,
                              const char *who)
{
    if (!W) return fail(SOM_ERR_INVALID_ARG, "%s: W is NULL", who);
    if (V < 1 || V >= INT32_MAX || E < 1 || E * E > SOM_MAX_NEURONS)
        return fail(SOM_ERR_INVALID_ARG, "%s: need 1 <= V < 2^31-1 and 1 <= E*E <= %d", who, SOM_MAX_NEURONS);
    if (N < 0 || N >= INT32_MAX || nnz < 0 || nnz > INT32_MAX)
        return fail(SOM_ERR_INVALID_ARG, "%s: N or nnz out of range", who);
    if (radius < 1) return fail(SOM_ERR_INVALID_ARG, "%s: radius must be >= 1 (got %d)", who, (int)radius);
    if (chunk_features < 0) return fail(SOM_ERR_INVALID_ARG, "%s: chunk_features must be >= 0", who);
    if (N > 0 && (!row_ptr || !bmu || (nnz > 0 && !col_idx))) return fail(SOM_ERR_INVALID_ARG, "%s: null pointer", who);
    som_status st = check_book(b, who);
    if (st != SOM_OK) return st;
    const int64_t M = E * E;
    const int64_t chunk = chunk_features == 0 || chunk_features > V ? V : chunk_features;
    const som::UpdateLayout L = som::update_layout(M, N, chunk);
    if (!workspace) return fail(SOM_ERR_WORKSPACE, "%s: workspace is NULL", who);
    if (reinterpret_cast<uintptr_t>(workspace) & 255) return fail(SOM_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    if (workspace_bytes < L.total)
        return fail(SOM_ERR_WORKSPACE, "%s: workspace holds %zu bytes, the update needs %zu", who, workspace_bytes,
                    L.total);
    if (N == 0) return ok();  // no sample: every unit keeps its prototype
    char *w = static_cast<char *>(workspace);
    som::UpdateBuffers ub;
    ub.flags = reinterpret_cast<uint32_t *>(w + L.flags);
    ub.den_cnt = reinterpret_cast<int32_t *>(w + L.den_cnt);
    ub.sup_row = reinterpret_cast<int32_t *>(w + L.sup_row);
    ub.sup = reinterpret_cast<int32_t *>(w + L.sup);
    ub.den_a = reinterpret_cast<float *>(w + L.den_a);
    ub.den_b = reinterpret_cast<float *>(w + L.den_b);
    ub.den_blur = reinterpret_cast<float *>(w + L.den_blur);
    ub.start = reinterpret_cast<int32_t *>(w + L.start);
    ub.cursor = reinterpret_cast<int32_t *>(w + L.cursor);
    ub.slot = reinterpret_cast<int32_t *>(w + L.slot);
    ub.hunit = reinterpret_cast<int32_t *>(w + L.hunit);
    ub.order = reinterpret_cast<int32_t *>(w + L.order);
    ub.cnt = reinterpret_cast<int32_t *>(w + L.cnt);
    ub.a = reinterpret_cast<float *>(w + L.a);
    ub.b = reinterpret_cast<float *>(w + L.b);
    hipError_t e = som::launch_update(b.f16, W, V, E, row_ptr, col_idx, N, nnz, bmu, radius, chunk, ub,
                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

som_status som_update(float *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx, int64_t N,
                      int64_t nnz, const int32_t *bmu, int32_t radius, int64_t chunk_features, void *workspace,
                      size_t workspace_bytes, void *stream)
{
    return update_impl(Book{W, false}, W, V, E, row_ptr, col_idx, N, nnz, bmu, radius, chunk_features, workspace,
                       workspace_bytes, stream, "som_update");
}

som_status som_update_f16(uint16_t *W, int64_t V, int64_t E, const int32_t *row_ptr, const int32_t *col_idx, int64_t N,
                          int64_t nnz, const int32_t *bmu, int32_t radius, int64_t chunk_features, void *workspace,
                          size_t workspace_bytes, void *stream)
{
    return update_impl(Book{W, true}, W, V, E, row_ptr, col_idx, N, nnz, bmu, radius, chunk_features, workspace,
                       workspace_bytes, stream, "som_update_f16");
}

double som_sigma(int32_t epoch, double sigma0, double sigma_min, double rate)
{
    if (epoch < 1) epoch = 1;
    return sigma_min + (sigma0 - sigma_min) * exp(-rate * (double)(epoch - 1));
}

int32_t som_radius(double sigma)
{
    if (!(sigma >= 1.0)) return 1;  // also NaN
    const double r = floor(sigma + 0.5);
    return r > (double)INT32_MAX ? INT32_MAX : (int32_t)r;
}

som_status som_validate_csr_host(const int32_t *row_ptr, const int32_t *col_idx, int64_t N, int64_t V)
{
    if (N < 0 || V < 1 || V >= INT32_MAX) return fail(SOM_ERR_INVALID_ARG, "need N >= 0 and 1 <= V < 2^31-1");
    if (!row_ptr) return fail(SOM_ERR_INVALID_ARG, "row_ptr is NULL");
    // col_idx is the base the offsets index: a negative offset would name ids before it
    if (row_ptr[0] < 0) return fail(SOM_ERR_BAD_CSR, "row_ptr[0] is negative (%d)", row_ptr[0]);
    for (int64_t s = 0; s < N; ++s)
        if (row_ptr[s + 1] < row_ptr[s])
            return fail(SOM_ERR_BAD_CSR, "row %lld: row_ptr decreases (%d -> %d)", (long long)s, row_ptr[s],
                        row_ptr[s + 1]);
    if (row_ptr[N] > row_ptr[0] && !col_idx) return fail(SOM_ERR_INVALID_ARG, "col_idx is NULL");
    for (int64_t s = 0; s < N; ++s) {
        for (int64_t p = row_ptr[s]; p < row_ptr[s + 1]; ++p) {
            const int32_t id = col_idx[p];
            if (id < 0 || id >= V)
                return fail(SOM_ERR_BAD_CSR, "row %lld: feature id %d outside [0, %lld)", (long long)s, id,
                            (long long)V);
            if (p > row_ptr[s] && id <= col_idx[p - 1])
                return fail(SOM_ERR_BAD_CSR, "row %lld: ids not strictly ascending (%d after %d)", (long long)s, id,
                            col_idx[p - 1]);
        }
    }
    return ok();
}

const char *som_last_error(void) { return g_err; }

}  // extern "C"
