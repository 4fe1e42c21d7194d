// C ABI of the IsoQuant stage-1 library (declared in include/isoquant.h):
// argument validation, the parameter handle, and kernel launches.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "isoq_internal.h"
#include "isoq_scores_generic.h"
#include "isoquant.h"

struct isoq_params {
    int variant, d, bits, n_sets;
    int device;
    float *dparams;                 // device, [n_sets][slots_per_set][params_per_slot], then the LUT
    size_t lut_offset;              // floats from dparams to the magnitude LUT (0: none)
    size_t mfma_offset;             // floats from dparams to the matrix-core parameters (0: none)
    int lut_cells;
    float lut_inv_h;
    std::vector<float> exported;    // unit parameters as used (Table 1 layout)
    float levels[16], thresholds[15];
};

struct isoq_sketch {
    int variant, d, n_sets, m;
    int device;
    uint16_t *dfrag;                // device, [n_sets][m/16][d/32][64][8] fp16 of S' = S T^{-1}
    float *dS;                      // device, [m][d] fp32 of S (query side)
    std::vector<float> S;           // host copy of S as used
};

namespace {

using namespace isoq;

// Text of the last HIP error seen by a call on this thread.
thread_local char g_last_hip_error[160] = "";

isoq_status hip_fail(hipError_t e, const char *where, isoq_status st = ISOQ_E_HIP)
{
    std::snprintf(g_last_hip_error, sizeof g_last_hip_error, "%s: %s (%d)", where,
                  hipGetErrorString(e), (int)e);
    return st;
}

bool valid_variant(int v) { return v == ISOQ_FULL || v == ISOQ_FAST || v == ISOQ_PLANAR2D || v == ISOQ_BLOCK8; }
// Widths of the tuned kernels (every entry point); other widths up to
// kGenericMaxD have quantize, dequantize and round trip only.
bool tuned_d(int d) { return d == 64 || d == 128 || d == 256 || d == 512; }
// widths of the decoding calls (append, logits): the tuned ones and three
// common attention head widths
bool decode_d(int d) { return tuned_d(d) || d == 80 || d == 96 || d == 160 || d == 192; }
// (d, m) of the stage-2 sketch: m = 64 or 128 sign bits at the decoding
// widths up to 192, m = 64 at 256 and 512 (the staged projection, m d fp16,
// has to fit the LDS next to the error tiles)
bool sketch_shape(int d, int m) { return decode_d(d) && (m == 64 || (m == 128 && d <= 192)); }
// fp16 rows at the head widths 80, 96, 160 and 192 take the packed-row
// kernels (rows of a group back to back across the wave; with 3 bits a row
// spans a multiple of 4 lanes, or 10 lanes at d = 80 with one chunk per lane)
bool packed_decode(int d, int bits, bool f16)
{
    const PackedShape ps = packed_shape(d, bits, f16);
    const int lanes = ps.rows > 0 ? d / (8 * ps.chunks) : 0;
    return !tuned_d(d) && decode_d(d) && f16 && ps.rows > 0 &&
           (bits != 3 || lanes % 4 == 0 || (ps.chunks == 1 && lanes % 2 == 0));
}
bool supported_d(int d) { return d >= 1 && d <= kGenericMaxD; }
bool supported_bits(int b) { return b >= 2 && b <= 4; }
bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

isoq_status check_common(const isoq_params *p, int dtype, int64_t n, int64_t rows_per_set)
{
    if (!p)
        return ISOQ_E_NULL;
    if (dtype != ISOQ_F32 && dtype != ISOQ_F16)
        return ISOQ_E_INVALID;
    if (n < 0 || rows_per_set < 1)
        return ISOQ_E_INVALID;
    return ISOQ_OK;
}

isoq_status check_device(const isoq_params *p)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    return dev == p->device ? ISOQ_OK : ISOQ_E_DEVICE;
}

// Rows of one block of the tuned stage-1 kernels (a wave holds 512/d rows).
int64_t rows_per_block(const isoq_params *p)
{
    return (int64_t)(64 / (p->d / kCoordsPerLane)) * (kBlockThreads / 64) * kTileGroups;
}

size_t record_bytes(int variant, int d, int bits)
{
    return ((size_t)padded_width(variant, d) * bits + 7) / 8;
}

// Per-handle kernel arguments: codebook halves, parameters, lookup table.
void fill_args(const isoq_params *p, KArgs &a)
{
    const int H = 1 << (p->bits - 1);
    for (int k = 0; k < H; k++)
        a.lev_pos[k] = p->levels[H + k];
    for (int k = 0; k + 1 < H; k++)
        a.thr_pos[k] = p->thresholds[H + k];
    for (int k = 0; k < 2 * H; k++)
        a.lev_all[k] = p->levels[k];
    a.params = p->dparams;
    a.n_sets = p->n_sets;
    a.lut = p->lut_offset ? p->dparams + p->lut_offset : nullptr;
    a.mfma = p->mfma_offset ? reinterpret_cast<const uint32_t *>(p->dparams + p->mfma_offset) : nullptr;
    a.lut_inv_h = p->lut_inv_h;
    a.lut_cells = p->lut_cells;
}

isoq_status launch(const void *fn, dim3 grid, void **args, void *stream, int threads = kBlockThreads)
{
    hipError_t e = hipLaunchKernel(fn, grid, dim3(threads), args, 0, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return hip_fail(e, "hipLaunchKernel");
    e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "after hipLaunchKernel");
    return ISOQ_OK;
}

const void *packed_kernel(int variant, int bits, int mode, int chunks, int cache_lp = -1)
{
    switch (variant) {
    case VAR_FULL: return packed_kernel_full(bits, mode, chunks, cache_lp);
    case VAR_FAST: return packed_kernel_fast(bits, mode, chunks, cache_lp);
    case VAR_PLANAR2D: return packed_kernel_2d(bits, mode, chunks, cache_lp);
    case VAR_BLOCK8: return packed_kernel_8d(bits, mode, chunks, cache_lp);
    }
    return nullptr;
}

// Widths outside {64, 128, 256, 512}: the packed-row kernels where a shape
// has them (not for append, whose packed kernel has a grid of its own), else
// the generic kernels.
isoq_status run_generic(const isoq_params *p, int dtype, int mode, KArgs &a, void *stream)
{
    // the generic kernels' slots: 4 coordinates (a 2-D row of 4k + 2
    // coordinates ends in a half slot), or 8 for 8-D blocks
    const int sw = p->variant == VAR_BLOCK8 ? 8 : 4;
    const int slots = (padded_width(p->variant, p->d) + sw - 1) / sw;
    if (slots < 1)
        return ISOQ_E_UNSUPPORTED;
    const bool f16 = dtype == ISOQ_F16;
    const PackedShape ps = packed_shape(p->d, p->bits, f16);
    const bool pairs = sw == 4 && f16 && p->d % 4 == 2;
    const int v = mode == MODE_APPEND ? 0 : ps.rows;
    const void *fn = v > 0 ? packed_kernel(p->variant, p->bits, mode, ps.chunks)
                     : p->variant == VAR_FULL   ? generic_kernel_full(slots, p->bits, f16, mode, pairs)
                     : p->variant == VAR_FAST   ? generic_kernel_fast(slots, p->bits, f16, mode, pairs)
                     : p->variant == VAR_BLOCK8 ? generic_kernel_8d(slots, p->bits, f16, mode, pairs)
                                                : generic_kernel_2d(slots, p->bits, f16, mode, pairs);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    // rows per block: packed, tiles of 4 waves of kTileGroups / chunks groups
    // of v rows; generic, 4 waves of their row groups
    const int64_t rpb = v > 0 ? (int64_t)v * (kBlockThreads / 64) * (kTileGroups / ps.chunks) *
                                    packed_tiles_per_block(p->variant, ps.chunks)
                              : (int64_t)generic_rows_per_wave(slots, sw, f16) * (kBlockThreads / 64);
    const int64_t blocks = (a.n + rpb - 1) / rpb;
    if (blocks > 0x7FFFFFFF)
        return ISOQ_E_UNSUPPORTED;
    fill_args(p, a);
    a.g_d = p->d;
    a.g_pw = padded_width(p->variant, p->d);
    a.g_slots = slots;
    a.g_rec = (int32_t)record_bytes(p->variant, p->d, p->bits);
    a.g_vec = p->d % sw == 0;
    a.g_rows = v;
    a.g_block_set = p->n_sets == 1 || (v > 0 && a.rows_per_set % rpb == 0);
    a.g_set_stride = (int64_t)slots_per_set(p->variant, p->d) * params_per_slot(p->variant);
    void *args[] = {&a};
    return launch(fn, dim3((unsigned)blocks), args, stream);
}

isoq_status run(const isoq_params *p, int dtype, int mode, KArgs &a, void *stream)
{
    if (!tuned_d(p->d))
        return run_generic(p, dtype, mode, a, stream);
    const bool f16 = dtype == ISOQ_F16;
    const int64_t rpb = rows_per_block(p);
    const bool generic = p->n_sets > 1 && (a.rows_per_set % rpb) != 0;
    // fp16 encoders whose blocks each have one set rotate on the matrix cores
    // (the decoder is the same in both layouts); so do rows with one set each
    // in turn (rows_per_set = 1), as n_sets streams of one set each
    const bool quad = f16 && quad_layout(p->variant, p->d, p->bits) && mode != MODE_DEQUANTIZE;
    if (quad && generic && a.rows_per_set == 1) {
        const int64_t per_stream = (a.n + p->n_sets - 1) / p->n_sets;
        const int64_t tiles = (per_stream + rpb - 1) / rpb;
        if (tiles <= 65535) {
            const void *fn = kernel_m_for(p->variant, p->d, p->bits,
                                          mode == MODE_ROUNDTRIP ? MODE_STREAMS_ROUNDTRIP : MODE_STREAMS_QUANTIZE);
            if (!fn)
                return ISOQ_E_UNSUPPORTED;
            fill_args(p, a);
            void *args[] = {&a};
            return launch(fn, dim3((unsigned)p->n_sets, (unsigned)tiles), args, stream);
        }
    }
    const void *fn = quad && !generic ? kernel_m_for(p->variant, p->d, p->bits, mode)
                                      : kernel_for(p->variant, p->d, p->bits, f16, generic, mode);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    const int64_t blocks = (a.n + rpb - 1) / rpb;
    if (blocks > 0x7FFFFFFF)
        return ISOQ_E_UNSUPPORTED;
    fill_args(p, a);
    void *args[] = {&a};
    return launch(fn, dim3((unsigned)blocks), args, stream);
}

}  // namespace

extern "C" {

const char *isoq_last_hip_error(void) { return g_last_hip_error; }

const char *isoq_status_string(isoq_status s)
{
    switch (s) {
    case ISOQ_OK: return "ok";
    case ISOQ_E_INVALID: return "invalid argument";
    case ISOQ_E_UNSUPPORTED:
        return "unsupported shape (d in 1..1024, bits in {2,3,4}; the sketch and the corrected logits need d "
               "in {64,80,96,128,160,192,256,512}) or size limit";
    case ISOQ_E_NULL: return "null pointer";
    case ISOQ_E_ALIGN: return "misaligned pointer";
    case ISOQ_E_HIP: return "HIP runtime error";
    case ISOQ_E_NOMEM: return "out of memory";
    case ISOQ_E_DEVICE: return "current device differs from the handle's device";
    }
    return "unknown status";
}

size_t isoq_packed_bytes(int d, int bits)
{
    if (d < 1 || bits < 1 || bits > 8)
        return 0;
    return ((size_t)d * bits + 7) / 8;
}

size_t isoq_record_bytes(int variant, int d, int bits)
{
    if (!valid_variant(variant) || d < 1 || bits < 1 || bits > 8)
        return 0;
    return record_bytes(variant, d, bits);
}

size_t isoq_raw_params_per_set(int variant, int d)
{
    if (!valid_variant(variant) || d < 1)
        return 0;
    return raw_per_set(variant, d);
}

size_t isoq_export_params_per_set(int variant, int d)
{
    if (!valid_variant(variant) || d < 1)
        return 0;
    return export_per_set(variant, d);
}

isoq_status isoq_codebook_lloyd(int bits, int d, int iters, double *levels_out)
{
    if (!levels_out)
        return ISOQ_E_NULL;
    if (d < 1 || iters < 0 || bits < 1 || bits > 8)
        return ISOQ_E_INVALID;
    if (!supported_bits(bits))
        return ISOQ_E_UNSUPPORTED;
    return lloyd_levels(bits, 1.0 / std::sqrt((double)d), iters, levels_out) ? ISOQ_OK : ISOQ_E_INVALID;
}

isoq_status isoq_rotation_draws(int variant, int d, int n_sets, uint64_t seed, double *out)
{
    if (!out)
        return ISOQ_E_NULL;
    if (!valid_variant(variant) || d < 1 || n_sets < 1)
        return ISOQ_E_INVALID;
    seeded_draws(variant, d, n_sets, seed, out);
    return ISOQ_OK;
}

isoq_status isoq_params_init(isoq_params **out, int variant, int d, int bits, int n_sets,
                             const double *rot_host, const double *codebook_host, uint64_t seed)
{
    if (!out)
        return ISOQ_E_NULL;
    *out = nullptr;
    if (!valid_variant(variant) || d < 1 || bits < 1 || bits > 8 || n_sets < 1)
        return ISOQ_E_INVALID;
    if (!supported_d(d) || !supported_bits(bits))
        return ISOQ_E_UNSUPPORTED;

    const int K = 1 << bits;
    double lev[16];
    if (codebook_host) {
        double mx = 0;
        for (int k = 0; k < K; k++) {
            if (!std::isfinite(codebook_host[k]))
                return ISOQ_E_INVALID;
            mx = std::max(mx, std::fabs(codebook_host[k]));
        }
        for (int k = 0; k + 1 < K; k++)
            if (!(codebook_host[k] < codebook_host[k + 1]))
                return ISOQ_E_INVALID;
        for (int k = 0; k < K / 2; k++) {
            if (std::fabs(codebook_host[k] + codebook_host[K - 1 - k]) > 1e-6 * mx)
                return ISOQ_E_INVALID;
            const double m = 0.5 * (codebook_host[K - 1 - k] - codebook_host[k]);
            lev[k] = -m;
            lev[K - 1 - k] = m;
        }
    } else if (!lloyd_levels(bits, 1.0 / std::sqrt((double)d), 200, lev)) {
        return ISOQ_E_INVALID;
    }

    std::vector<double> drawn;
    const double *raw = rot_host;
    if (!raw) {
        try {
            drawn.resize((size_t)n_sets * raw_per_set(variant, d));
        } catch (const std::bad_alloc &) {
            return ISOQ_E_NOMEM;
        }
        seeded_draws(variant, d, n_sets, seed, drawn.data());
        raw = drawn.data();
    }
    isoq_params *p = new (std::nothrow) isoq_params();
    if (!p)
        return ISOQ_E_NOMEM;
    p->variant = variant;
    p->d = d;
    p->bits = bits;
    p->n_sets = n_sets;
    p->dparams = nullptr;
    std::vector<float> layout;
    try {
        if (!build_rotation(variant, d, n_sets, raw, p->exported, layout)) {
            delete p;
            return ISOQ_E_INVALID;
        }
    } catch (const std::bad_alloc &) {
        delete p;
        return ISOQ_E_NOMEM;
    }
    for (int k = 0; k < K; k++)
        p->levels[k] = (float)lev[k];
    for (int k = 0; k + 1 < K; k++)
        p->thresholds[k] = (float)(0.5 * (lev[k] + lev[k + 1]));
    p->thresholds[K / 2 - 1] = 0.0f;
    p->lut_offset = 0;
    p->lut_cells = 0;
    p->lut_inv_h = 0.f;
    if (bits == 4) {
        // thresholds and levels of the positive half, in fp32 as the kernels use them
        const int H = K / 2;
        double tau[8], levp[8], inv_h = 0;
        for (int i = 0; i + 1 < H; i++)
            tau[i] = (double)p->thresholds[H + i];
        for (int i = 0; i < H; i++)
            levp[i] = (double)p->levels[H + i];
        std::vector<LutEntry> lut;
        if (!build_magnitude_lut(H, tau, levp, &inv_h, lut)) {
            delete p;
            return ISOQ_E_UNSUPPORTED;
        }
        p->lut_offset = layout.size();
        p->lut_cells = (int)lut.size();
        p->lut_inv_h = (float)inv_h;
        const float *f = reinterpret_cast<const float *>(lut.data());
        layout.insert(layout.end(), f, f + 4 * lut.size());
    }
    // the matrix-core encoders' fp16 (hi, lo) matrix rows, after the rest
    // (16-byte aligned: every part above is a multiple of 4 floats)
    p->mfma_offset = 0;
    if (quad_layout(variant, d, bits)) {
        const size_t per_set = mfma_bytes_per_set(variant, d);
        std::vector<uint16_t> mf;
        try {
            mf.resize((size_t)n_sets * per_set / 2);
        } catch (const std::bad_alloc &) {
            delete p;
            return ISOQ_E_NOMEM;
        }
        const size_t slots = (size_t)slots_per_set(variant, d) * params_per_slot(variant);
        for (int s = 0; s < n_sets; s++)
            build_mfma_params(variant, d, layout.data() + s * slots, mf.data() + s * per_set / 2);
        while (layout.size() % 4)
            layout.push_back(0.f);
        p->mfma_offset = layout.size();
        const float *f = reinterpret_cast<const float *>(mf.data());
        layout.insert(layout.end(), f, f + mf.size() / 2);
    }

    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return hip_fail(e, "hipGetDevice");
    }
    const size_t bytes = layout.size() * sizeof(float);
    e = hipMalloc(reinterpret_cast<void **>(&p->dparams), bytes);
    if (e != hipSuccess) {
        delete p;
        return hip_fail(e, "hipMalloc", e == hipErrorOutOfMemory ? ISOQ_E_NOMEM : ISOQ_E_HIP);
    }
    e = hipMemcpy(p->dparams, layout.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(p->dparams);
        delete p;
        return hip_fail(e, "hipMemcpy");
    }
    *out = p;
    return ISOQ_OK;
}

isoq_status isoq_params_destroy(isoq_params *p)
{
    if (!p)
        return ISOQ_OK;
    isoq_status st = ISOQ_OK;
    if (p->dparams) {
        int prev = -1;
        (void)hipGetDevice(&prev);
        if (prev != p->device)
            (void)hipSetDevice(p->device);
        if (hipFree(p->dparams) != hipSuccess)
            st = ISOQ_E_HIP;
        if (prev >= 0 && prev != p->device)
            (void)hipSetDevice(prev);
    }
    delete p;
    return st;
}

isoq_status isoq_params_export(const isoq_params *p, float *rot_out, float *levels_out,
                               float *thresholds_out)
{
    if (!p)
        return ISOQ_E_NULL;
    const int K = 1 << p->bits;
    if (rot_out)
        std::memcpy(rot_out, p->exported.data(), p->exported.size() * sizeof(float));
    if (levels_out)
        std::memcpy(levels_out, p->levels, K * sizeof(float));
    if (thresholds_out)
        std::memcpy(thresholds_out, p->thresholds, (K - 1) * sizeof(float));
    return ISOQ_OK;
}

isoq_status isoq_params_info(const isoq_params *p, int *variant, int *d, int *bits, int *n_sets)
{
    if (!p)
        return ISOQ_E_NULL;
    if (variant)
        *variant = p->variant;
    if (d)
        *d = p->d;
    if (bits)
        *bits = p->bits;
    if (n_sets)
        *n_sets = p->n_sets;
    return ISOQ_OK;
}

isoq_status isoq_roundtrip(const isoq_params *p, int dtype, const void *x, int64_t n,
                           int64_t rows_per_set, void *x_hat, void *stream)
{
    isoq_status st = check_common(p, dtype, n, rows_per_set);
    if (st != ISOQ_OK)
        return st;
    if (n == 0)
        return ISOQ_OK;
    if (!x || !x_hat)
        return ISOQ_E_NULL;
    if (!aligned(x, 16) || !aligned(x_hat, 16))
        return ISOQ_E_ALIGN;
    if ((st = check_device(p)) != ISOQ_OK)
        return st;
    KArgs a{};
    a.x = x;
    a.y = x_hat;
    a.n = n;
    a.rows_per_set = rows_per_set;
    return run(p, dtype, MODE_ROUNDTRIP, a, stream);
}

isoq_status isoq_quantize(const isoq_params *p, int dtype, const void *x, int64_t n,
                          int64_t rows_per_set, uint8_t *idx_packed, float *norms, void *stream)
{
    isoq_status st = check_common(p, dtype, n, rows_per_set);
    if (st != ISOQ_OK)
        return st;
    if (n == 0)
        return ISOQ_OK;
    if (!x || !idx_packed || !norms)
        return ISOQ_E_NULL;
    if (!aligned(x, 16) || !aligned(idx_packed, 4) || !aligned(norms, 4))
        return ISOQ_E_ALIGN;
    if ((st = check_device(p)) != ISOQ_OK)
        return st;
    KArgs a{};
    a.x = x;
    a.rec_out = idx_packed;
    a.norms_out = norms;
    a.n = n;
    a.rows_per_set = rows_per_set;
    return run(p, dtype, MODE_QUANTIZE, a, stream);
}

isoq_status isoq_dequantize(const isoq_params *p, int dtype, const uint8_t *idx_packed,
                            const float *norms, int64_t n, int64_t rows_per_set, void *x_hat,
                            void *stream)
{
    isoq_status st = check_common(p, dtype, n, rows_per_set);
    if (st != ISOQ_OK)
        return st;
    if (n == 0)
        return ISOQ_OK;
    if (!idx_packed || !norms || !x_hat)
        return ISOQ_E_NULL;
    if (!aligned(x_hat, 16) || !aligned(idx_packed, 4) || !aligned(norms, 4))
        return ISOQ_E_ALIGN;
    if ((st = check_device(p)) != ISOQ_OK)
        return st;
    KArgs a{};
    a.y = x_hat;
    a.rec_in = idx_packed;
    a.norms_in = norms;
    a.n = n;
    a.rows_per_set = rows_per_set;
    return run(p, dtype, MODE_DEQUANTIZE, a, stream);
}

isoq_status isoq_kv_append(const isoq_params *pk, const isoq_params *pv, int dtype,
                           const void *k_new, const void *v_new, const int64_t *slot_mapping,
                           int64_t n_tokens, int n_heads, uint8_t *k_idx, float *k_rho,
                           uint8_t *v_idx, float *v_rho, int64_t n_blocks, int block_size,
                           void *stream)
{
    if (!pk)
        return ISOQ_E_NULL;
    if (dtype != ISOQ_F32 && dtype != ISOQ_F16)
        return ISOQ_E_INVALID;
    if (n_tokens < 0 || n_heads < 1 || block_size < 1 || n_blocks < 0)
        return ISOQ_E_INVALID;
    const bool has_v = pv || v_new || v_idx || v_rho;
    if (has_v && !(pv && v_new && v_idx && v_rho))
        return ISOQ_E_NULL;
    if (has_v && (pv->variant != pk->variant || pv->d != pk->d || pv->bits != pk->bits ||
                  pv->device != pk->device))
        return ISOQ_E_INVALID;
    // fp16 rows at d = 80, 96, 160 and 192 use the packed-row kernels (rows
    // of a group back to back across the wave; with 3 bits a row spans a
    // multiple of 4 lanes, or 10 lanes at d = 80 with one chunk per lane)
    // other shapes (fp32 rows, other widths) use the generic kernels
    const PackedShape ps = packed_shape(pk->d, pk->bits, true);
    const bool packed = packed_decode(pk->d, pk->bits, dtype == ISOQ_F16);
    const bool generic = !tuned_d(pk->d) && !packed;
    if ((pk->n_sets != 1 && pk->n_sets != n_heads) || (has_v && pv->n_sets != 1 && pv->n_sets != n_heads))
        return ISOQ_E_INVALID;
    if (n_tokens > 0x7FFFFFFF / n_heads || n_blocks > 0x7FFFFFFF / block_size)
        return ISOQ_E_UNSUPPORTED;
    if (n_tokens == 0 || n_blocks == 0)
        return ISOQ_OK;
    if (!k_new || !slot_mapping || !k_idx || !k_rho)
        return ISOQ_E_NULL;
    if (!aligned(k_new, 16) || !aligned(slot_mapping, 8) || !aligned(k_idx, 4) || !aligned(k_rho, 4))
        return ISOQ_E_ALIGN;
    if (has_v && (!aligned(v_new, 16) || !aligned(v_idx, 4) || !aligned(v_rho, 4)))
        return ISOQ_E_ALIGN;
    isoq_status st = check_device(pk);
    if (st != ISOQ_OK)
        return st;
    if (generic) {
        // one launch per tensor over the n_tokens * n_heads (token, head)
        // rows of its input, row t n_heads + h with set h (or set 0)
        for (int t = 0; t < (has_v ? 2 : 1); t++) {
            KArgs a{};
            a.x = t == 0 ? k_new : v_new;
            a.rec_out = t == 0 ? k_idx : v_idx;
            a.norms_out = t == 0 ? k_rho : v_rho;
            a.n = n_tokens * n_heads;
            a.rows_per_set = 1;
            a.slots = slot_mapping;
            a.n_slots = n_blocks * block_size;
            a.n_heads = (uint32_t)n_heads;
            a.block_size = (uint32_t)block_size;
            a.div_block = make_fastdiv((uint32_t)block_size);
            if ((st = run_generic(t == 0 ? pk : pv, dtype, MODE_APPEND, a, stream)) != ISOQ_OK)
                return st;
        }
        return ISOQ_OK;
    }
    // one kernel for both tensors; block (x, y, z) = (head, token range, K|V)
    const bool quad = dtype == ISOQ_F16 && quad_layout(pk->variant, pk->d, pk->bits);
    const int64_t rec_b = (int64_t)record_bytes(pk->variant, pk->d, pk->bits);
    const int cache_lp = rec_b % 16 == 0 ? 4 : rec_b % 8 == 0 ? 3 : -1;   // cache_piece
    const void *fn = packed ? packed_kernel(pk->variant, pk->bits, MODE_APPEND, ps.chunks, cache_lp)
                     : quad ? kernel_m_for(pk->variant, pk->d, pk->bits, MODE_APPEND)
                            : kernel_for(pk->variant, pk->d, pk->bits, dtype == ISOQ_F16, false, MODE_APPEND);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    // tokens per block: 4 waves of kTileGroups (packed: kTileGroups / chunks)
    // row groups
    const int64_t rpb = packed ? (int64_t)ps.rows * (kBlockThreads / 64) * (kTileGroups / ps.chunks)
                               : rows_per_block(pk);
    const int64_t blocks = (n_tokens + rpb - 1) / rpb;
    if (blocks > 65535)
        return ISOQ_E_UNSUPPORTED;
    KArgs ak{}, av{};
    for (int t = 0; t < (has_v ? 2 : 1); t++) {
        KArgs &a = t == 0 ? ak : av;
        fill_args(t == 0 ? pk : pv, a);
        a.x = t == 0 ? k_new : v_new;
        a.rec_out = t == 0 ? k_idx : v_idx;
        a.norms_out = t == 0 ? k_rho : v_rho;
        a.n = n_tokens;
        a.rows_per_set = 1;
        a.slots = slot_mapping;
        a.n_slots = n_blocks * block_size;
        a.n_heads = (uint32_t)n_heads;
        a.block_size = (uint32_t)block_size;
        a.div_block = make_fastdiv((uint32_t)block_size);
        if (packed) {
            a.g_d = pk->d;
            a.g_rows = ps.rows;
            a.g_set_stride = (int64_t)slots_per_set(pk->variant, pk->d) * params_per_slot(pk->variant);
        }
    }
    void *args[] = {&ak, &av};
    return launch(fn, dim3((unsigned)n_heads, (unsigned)blocks, has_v ? 2 : 1), args, stream);
}

}  // extern "C"

namespace {

// isoq_kv_scores at widths without a tuned logit kernel (arguments checked
// by kv_scores): one workgroup per (query head, chunk, sequence).
isoq_status kv_scores_generic(const isoq_params *pk, int dtype, const void *q, int n_seqs, int n_q_heads,
                              int n_kv_heads, const uint8_t *k_idx, const float *k_rho, int64_t n_blocks,
                              int block_size, const int32_t *block_table, int max_blocks_per_seq,
                              const int32_t *seq_lens, float scale, float *scores, int64_t max_len,
                              int64_t max_pos, void *stream)
{
    const void *fn = generic_score_kernel_for(pk->variant, pk->bits, dtype == ISOQ_F16);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    const int sw = pk->variant == VAR_BLOCK8 ? 8 : 4;
    GenScoreShape g{};
    g.d = pk->d;
    g.slots = (padded_width(pk->variant, pk->d) + sw - 1) / sw;
    g.rec = (int32_t)record_bytes(pk->variant, pk->d, pk->bits);
    g.rec_lp = g.rec % 16 == 0 ? 4 : g.rec % 8 == 0 ? 3 : -1;   // cache_piece
    g.set_stride = (int64_t)slots_per_set(pk->variant, pk->d) * params_per_slot(pk->variant);
    SArgs a{};
    a.q = q;
    a.k_idx = k_idx;
    a.k_rho = k_rho;
    a.block_table = block_table;
    a.seq_lens = seq_lens;
    a.scores = scores;
    a.params = pk->dparams;
    a.max_len = max_len;
    a.n_blocks = n_blocks;
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.group = n_q_heads / n_kv_heads;
    a.block_size = block_size;
    a.max_blocks = max_blocks_per_seq;
    a.n_sets = pk->n_sets;
    a.scale = scale;
    a.div_block = make_fastdiv((uint32_t)block_size);
    for (int k = 0; k < (1 << pk->bits); k++)
        a.lev_all[k] = pk->levels[k];
    void *args[] = {&a, &g};
    const dim3 grid((unsigned)n_q_heads, (unsigned)((max_pos + kScoreChunk - 1) / kScoreChunk), (unsigned)n_seqs);
    hipError_t e = hipLaunchKernel(fn, grid, dim3(256), args, generic_score_lds(g.slots, pk->variant),
                                   static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return hip_fail(e, "hipLaunchKernel");
    e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "after hipLaunchKernel");
    return ISOQ_OK;
}

// isoq_kv_scores and isoq_kv_scores_qjl (sk, k_signs, k_gamma non-NULL).
isoq_status kv_scores(const isoq_params *pk, const isoq_sketch *sk, int dtype, const void *q, int n_seqs,
                      int n_q_heads, int n_kv_heads, const uint8_t *k_idx, const float *k_rho,
                      const uint8_t *k_signs, const float *k_gamma, int64_t n_blocks, int block_size,
                      const int32_t *block_table, int max_blocks_per_seq, const int32_t *seq_lens, float scale,
                      float *scores, int64_t max_len, void *stream)
{
    if (!pk)
        return ISOQ_E_NULL;
    if (dtype != ISOQ_F32 && dtype != ISOQ_F16)
        return ISOQ_E_INVALID;
    if (n_seqs < 0 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 ||
        block_size < 1 || n_blocks < 0 || max_blocks_per_seq < 0 || max_len < 0 || !std::isfinite(scale))
        return ISOQ_E_INVALID;
    if (pk->n_sets != 1 && pk->n_sets != n_kv_heads)
        return ISOQ_E_INVALID;
    if (sk && (sk->variant != pk->variant || sk->d != pk->d || sk->n_sets != pk->n_sets ||
               sk->device != pk->device))
        return ISOQ_E_INVALID;
    // widths without a tuned logit kernel: the width-generic one (no sketch
    // exists at those widths)
    const bool generic = !decode_d(pk->d);
    if (generic && sk)
        return ISOQ_E_UNSUPPORTED;
    const int64_t max_pos = std::min<int64_t>(max_len, (int64_t)max_blocks_per_seq * block_size);
    if (n_seqs > 65535 || (int64_t)max_blocks_per_seq * block_size > 0x7FFFFFFF ||
        (max_pos + kScoreChunk - 1) / kScoreChunk > 65535)
        return ISOQ_E_UNSUPPORTED;
    if (n_seqs == 0 || max_pos == 0 || n_blocks == 0)
        return ISOQ_OK;
    if (!q || !k_idx || !k_rho || !block_table || !seq_lens || !scores)
        return ISOQ_E_NULL;
    if (sk && (!k_signs || !k_gamma))
        return ISOQ_E_NULL;
    if (!aligned(q, 16) || !aligned(k_idx, 16) || !aligned(k_rho, 4) || !aligned(block_table, 4) ||
        !aligned(seq_lens, 4) || !aligned(scores, 4))
        return ISOQ_E_ALIGN;
    if (sk && (!aligned(k_signs, 4) || !aligned(k_gamma, 4)))
        return ISOQ_E_ALIGN;
    isoq_status st = check_device(pk);
    if (st != ISOQ_OK)
        return st;
    const int group = n_q_heads / n_kv_heads;
    if (generic)
        return kv_scores_generic(pk, dtype, q, n_seqs, n_q_heads, n_kv_heads, k_idx, k_rho, n_blocks, block_size,
                                 block_table, max_blocks_per_seq, seq_lens, scale, scores, max_len, max_pos,
                                 stream);
    const ScoreKernel kern = sk ? score_qjl_kernel_for(pk->variant, pk->d, pk->bits, dtype == ISOQ_F16, group, sk->m)
                                : score_kernel_for(pk->variant, pk->d, pk->bits, dtype == ISOQ_F16, group);
    if (!kern.fn)
        return ISOQ_E_UNSUPPORTED;
    const void *fn = kern.fn;
    const size_t lds = kern.dyn_lds;
    int lds_max = 0;
    hipError_t e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, pk->device);
    if (e != hipSuccess)
        return hip_fail(e, "hipDeviceGetAttribute");
    if (lds > (size_t)lds_max)
        return ISOQ_E_UNSUPPORTED;
    if (lds > 65536) {
        e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess)
            return hip_fail(e, "hipFuncSetAttribute");
    }
    SArgs a{};
    a.q = q;
    a.k_idx = k_idx;
    a.k_rho = k_rho;
    a.block_table = block_table;
    a.seq_lens = seq_lens;
    a.scores = scores;
    a.params = pk->dparams;
    a.max_len = max_len;
    a.n_blocks = n_blocks;
    a.n_q_heads = n_q_heads;
    a.n_kv_heads = n_kv_heads;
    a.group = group;
    a.block_size = block_size;
    a.max_blocks = max_blocks_per_seq;
    a.n_sets = pk->n_sets;
    a.scale = scale;
    a.div_block = make_fastdiv((uint32_t)block_size);
    for (int k = 0; k < (1 << pk->bits); k++)
        a.lev_all[k] = pk->levels[k];
    if (sk) {
        a.qjl_S = sk->dS;
        a.k_signs = k_signs;
        a.k_gamma = k_gamma;
        a.qjl_scale = (float)((double)scale * std::sqrt(M_PI / 2.0) / sk->m);
    }
    void *args[] = {&a};
    const dim3 grid((unsigned)n_kv_heads, (unsigned)((max_pos + kScoreChunk - 1) / kScoreChunk), (unsigned)n_seqs);
    e = hipLaunchKernel(fn, grid, dim3(256), args, lds, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return hip_fail(e, "hipLaunchKernel");
    e = hipGetLastError();
    if (e != hipSuccess)
        return hip_fail(e, "after hipLaunchKernel");
    return ISOQ_OK;
}

}  // namespace

extern "C" {

isoq_status isoq_kv_scores(const isoq_params *pk, int dtype, const void *q, int n_seqs,
                           int n_q_heads, int n_kv_heads, const uint8_t *k_idx, const float *k_rho,
                           int64_t n_blocks, int block_size, const int32_t *block_table,
                           int max_blocks_per_seq, const int32_t *seq_lens, float scale,
                           float *scores, int64_t max_len, void *stream)
{
    return kv_scores(pk, nullptr, dtype, q, n_seqs, n_q_heads, n_kv_heads, k_idx, k_rho, nullptr, nullptr,
                     n_blocks, block_size, block_table, max_blocks_per_seq, seq_lens, scale, scores, max_len,
                     stream);
}

isoq_status isoq_kv_scores_qjl(const isoq_params *pk, const isoq_sketch *sk, int dtype, const void *q,
                               int n_seqs, int n_q_heads, int n_kv_heads, const uint8_t *k_idx,
                               const float *k_rho, const uint8_t *k_signs, const float *k_gamma,
                               int64_t n_blocks, int block_size, const int32_t *block_table,
                               int max_blocks_per_seq, const int32_t *seq_lens, float scale, float *scores,
                               int64_t max_len, void *stream)
{
    if (!sk)
        return ISOQ_E_NULL;
    return kv_scores(pk, sk, dtype, q, n_seqs, n_q_heads, n_kv_heads, k_idx, k_rho, k_signs, k_gamma, n_blocks,
                     block_size, block_table, max_blocks_per_seq, seq_lens, scale, scores, max_len, stream);
}

isoq_status isoq_sketch_init(isoq_sketch **out, const isoq_params *p, int m, const double *S_host,
                             uint64_t seed)
{
    if (!out)
        return ISOQ_E_NULL;
    *out = nullptr;
    if (!p)
        return ISOQ_E_NULL;
    if (m < 1)
        return ISOQ_E_INVALID;
    if (!sketch_shape(p->d, m) || p->variant == VAR_BLOCK8)
        return ISOQ_E_UNSUPPORTED;
    const int d = p->d;
    std::vector<double> S((size_t)m * d), Sp((size_t)m * d);
    if (S_host) {
        for (size_t i = 0; i < S.size(); i++) {
            if (!std::isfinite(S_host[i]))
                return ISOQ_E_INVALID;
            S[i] = S_host[i];
        }
    } else {
        seeded_projection(m, d, seed, S.data());
    }
    isoq_sketch *sk = new (std::nothrow) isoq_sketch();
    if (!sk)
        return ISOQ_E_NOMEM;
    sk->variant = p->variant;
    sk->d = d;
    sk->n_sets = p->n_sets;
    sk->m = m;
    sk->device = p->device;
    sk->dfrag = nullptr;
    sk->dS = nullptr;
    // S' = S T^{-1}: row i of S' is T applied to row i of S (T orthogonal),
    // with the handle's own fp32 rotation parameters; then fp16 in the order
    // lane l of k-step ks of column tile nt reads, S'[c][32 ks + 8 (l / 16) + i]
    // with c = (m/4) (r / 4) + 4 nt + r % 4 for the tile row r = l % 16 (the
    // coordinate order that leaves each lane of the projection with m/4
    // consecutive sign bits of one row); zero past column d, up to the
    // projection width dp (a multiple of 32)
    const int dp = qjl_proj_width(d);
    const int KS = dp / 32, NT = m / 16;
    const size_t per_set = (size_t)m * dp;
    std::vector<uint16_t> frag;
    try {
        sk->S.assign(S.begin(), S.end());
        frag.resize((size_t)p->n_sets * per_set);
    } catch (const std::bad_alloc &) {
        delete sk;
        return ISOQ_E_NOMEM;
    }
    for (size_t i = 0; i < S.size(); i++)
        sk->S[i] = (float)S[i];
    const size_t ex_per_set = export_per_set(p->variant, d);
    for (int set = 0; set < p->n_sets; set++) {
        rotate_rows_forward(p->variant, d, p->exported.data() + set * ex_per_set, S.data(), m, Sp.data());
        uint16_t *f = frag.data() + set * per_set;
        for (int nt = 0; nt < NT; nt++)
            for (int ks = 0; ks < KS; ks++)
                for (int l = 0; l < 64; l++)
                    for (int i = 0; i < 8; i++) {
                        const int r = l % 16, c = m / 4 * (r / 4) + 4 * nt + r % 4;
                        const int k = 32 * ks + 8 * (l / 16) + i;
                        const _Float16 h = k < d ? (_Float16)Sp[(size_t)c * d + k] : (_Float16)0.f;
                        uint16_t bits;
                        std::memcpy(&bits, &h, 2);
                        f[((size_t)(nt * KS + ks) * 64 + l) * 8 + i] = bits;
                    }
    }
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&sk->dfrag), frag.size() * 2);
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&sk->dS), sk->S.size() * sizeof(float));
    if (e == hipSuccess)
        e = hipMemcpy(sk->dfrag, frag.data(), frag.size() * 2, hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(sk->dS, sk->S.data(), sk->S.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        if (sk->dfrag)
            (void)hipFree(sk->dfrag);
        if (sk->dS)
            (void)hipFree(sk->dS);
        delete sk;
        return hip_fail(e, "isoq_sketch_init", e == hipErrorOutOfMemory ? ISOQ_E_NOMEM : ISOQ_E_HIP);
    }
    *out = sk;
    return ISOQ_OK;
}

isoq_status isoq_sketch_destroy(isoq_sketch *sk)
{
    if (!sk)
        return ISOQ_OK;
    isoq_status st = ISOQ_OK;
    int prev = -1;
    (void)hipGetDevice(&prev);
    if (prev != sk->device)
        (void)hipSetDevice(sk->device);
    if (sk->dfrag && hipFree(sk->dfrag) != hipSuccess)
        st = ISOQ_E_HIP;
    if (sk->dS && hipFree(sk->dS) != hipSuccess)
        st = ISOQ_E_HIP;
    if (prev >= 0 && prev != sk->device)
        (void)hipSetDevice(prev);
    delete sk;
    return st;
}

isoq_status isoq_sketch_export(const isoq_sketch *sk, int *m, float *S_out)
{
    if (!sk)
        return ISOQ_E_NULL;
    if (m)
        *m = sk->m;
    if (S_out)
        std::memcpy(S_out, sk->S.data(), sk->S.size() * sizeof(float));
    return ISOQ_OK;
}

// The packed-row kernels' geometry in the arguments (tpb: row tiles per
// block).
static void set_packed_args(const isoq_params *p, const PackedShape &ps, int64_t tpb, KArgs &a)
{
    a.g_d = p->d;
    a.g_rows = ps.rows;
    a.g_tpb = (int32_t)tpb;
    a.g_block_set = 1;
    a.g_set_stride = (int64_t)slots_per_set(p->variant, p->d) * params_per_slot(p->variant);
}

// isoq_quantize_qjl at the head widths 80, 96, 160 and 192: fp16 rows, one
// rotation set, packed-row kernels of kPackedQjlWaves waves; blocks walk runs
// of g_tpb row tiles.
static isoq_status quantize_qjl_packed(const isoq_params *p, const isoq_sketch *sk, int dtype, const void *x,
                                       int64_t n, uint8_t *idx_packed, float *norms, uint8_t *signs, float *gamma,
                                       void *stream)
{
    if (!packed_decode(p->d, p->bits, dtype == ISOQ_F16) || p->n_sets != 1)
        return ISOQ_E_UNSUPPORTED;
    if (n == 0)
        return ISOQ_OK;
    if (!x || !idx_packed || !norms || !signs || !gamma)
        return ISOQ_E_NULL;
    if (!aligned(x, 16) || !aligned(idx_packed, 4) || !aligned(norms, 4) || !aligned(signs, 4) ||
        !aligned(gamma, 4))
        return ISOQ_E_ALIGN;
    isoq_status st = check_device(p);
    if (st != ISOQ_OK)
        return st;
    const void *fn = packed_qjl_kernel_for(p->variant, p->d, p->bits, sk->m, false);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    const PackedShape ps = packed_shape(p->d, p->bits, true);
    const int64_t per_tile = (int64_t)ps.rows * kPackedQjlWaves * packed_groups(ps.rows, ps.chunks, true);
    const int64_t tiles = (n + per_tile - 1) / per_tile;
    const int64_t blocks0 = std::min<int64_t>(tiles, kQjlBlocks * 4 / kPackedQjlWaves);
    const int64_t tpb = (tiles + blocks0 - 1) / blocks0;
    const int64_t blocks = (tiles + tpb - 1) / tpb;
    if (tpb > 0x7FFFFFFF)
        return ISOQ_E_UNSUPPORTED;
    KArgs a{};
    fill_args(p, a);
    a.x = x;
    a.rec_out = idx_packed;
    a.norms_out = norms;
    a.n = n;
    a.rows_per_set = 1;
    a.qjl_frag = sk->dfrag;
    a.qjl_signs = signs;
    a.qjl_gamma = gamma;
    set_packed_args(p, ps, tpb, a);
    void *args[] = {&a};
    return launch(fn, dim3((unsigned)blocks), args, stream, 64 * kPackedQjlWaves);
}

isoq_status isoq_quantize_qjl(const isoq_params *p, const isoq_sketch *sk, int dtype, const void *x,
                              int64_t n, int64_t rows_per_set, uint8_t *idx_packed, float *norms,
                              uint8_t *signs, float *gamma, void *stream)
{
    isoq_status st = check_common(p, dtype, n, rows_per_set);
    if (st != ISOQ_OK)
        return st;
    if (!sk)
        return ISOQ_E_NULL;
    if (sk->variant != p->variant || sk->d != p->d || sk->n_sets != p->n_sets || sk->device != p->device)
        return ISOQ_E_INVALID;
    if (!tuned_d(p->d))
        return quantize_qjl_packed(p, sk, dtype, x, n, idx_packed, norms, signs, gamma, stream);
    // rows of one tile (a block's waves, kTileGroups groups each)
    const int waves = qjl_waves(sk->m, false, p->n_sets);
    const int64_t rpb = rows_per_block(p) / 4 * waves;
    if (p->n_sets > 1 && rows_per_set % rpb != 0)
        return ISOQ_E_UNSUPPORTED;
    if (n == 0)
        return ISOQ_OK;
    if (!x || !idx_packed || !norms || !signs || !gamma)
        return ISOQ_E_NULL;
    if (!aligned(x, 16) || !aligned(idx_packed, 4) || !aligned(norms, 4) || !aligned(signs, 4) ||
        !aligned(gamma, 4))
        return ISOQ_E_ALIGN;
    if ((st = check_device(p)) != ISOQ_OK)
        return st;
    const void *fn = qjl_kernel_for(p->variant, p->d, p->bits, dtype == ISOQ_F16, sk->m, false, waves);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    const int64_t tiles = (n + rpb - 1) / rpb;
    if (tiles > 0x7FFFFFFF)
        return ISOQ_E_UNSUPPORTED;
    // with one rotation set, blocks walk several tiles each (the projection is
    // staged once per block; kQjlBlocks 4-wave blocks or half as many 8-wave
    // ones); otherwise one block per tile keeps each block on its own set
    const int64_t blocks = p->n_sets == 1 ? std::min<int64_t>(tiles, kQjlBlocks * 4 / waves) : tiles;
    KArgs a{};
    fill_args(p, a);
    a.x = x;
    a.rec_out = idx_packed;
    a.norms_out = norms;
    a.n = n;
    a.rows_per_set = rows_per_set;
    a.qjl_frag = sk->dfrag;
    a.qjl_signs = signs;
    a.qjl_gamma = gamma;
    void *args[] = {&a};
    return launch(fn, dim3((unsigned)blocks), args, stream, 64 * waves);
}

isoq_status isoq_kv_append_qjl(const isoq_params *pk, const isoq_sketch *sk, int dtype, const void *k_new,
                               const int64_t *slot_mapping, int64_t n_tokens, int n_heads, uint8_t *k_idx,
                               float *k_rho, uint8_t *k_signs, float *k_gamma, int64_t n_blocks, int block_size,
                               void *stream)
{
    if (!pk || !sk)
        return ISOQ_E_NULL;
    if (dtype != ISOQ_F32 && dtype != ISOQ_F16)
        return ISOQ_E_INVALID;
    if (n_tokens < 0 || n_heads < 1 || block_size < 1 || n_blocks < 0)
        return ISOQ_E_INVALID;
    if (sk->variant != pk->variant || sk->d != pk->d || sk->n_sets != pk->n_sets || sk->device != pk->device)
        return ISOQ_E_INVALID;
    if (pk->n_sets != 1 && pk->n_sets != n_heads)
        return ISOQ_E_INVALID;
    if (n_tokens > 0x7FFFFFFF / n_heads || n_blocks > 0x7FFFFFFF / block_size)
        return ISOQ_E_UNSUPPORTED;
    if (n_tokens == 0 || n_blocks == 0)
        return ISOQ_OK;
    if (!k_new || !slot_mapping || !k_idx || !k_rho || !k_signs || !k_gamma)
        return ISOQ_E_NULL;
    if (!aligned(k_new, 16) || !aligned(slot_mapping, 8) || !aligned(k_idx, 4) || !aligned(k_rho, 4) ||
        !aligned(k_signs, 4) || !aligned(k_gamma, 4))
        return ISOQ_E_ALIGN;
    isoq_status st = check_device(pk);
    if (st != ISOQ_OK)
        return st;
    KArgs a{};
    fill_args(pk, a);
    a.x = k_new;
    a.rec_out = k_idx;
    a.norms_out = k_rho;
    a.n = n_tokens;
    a.rows_per_set = 1;
    a.slots = slot_mapping;
    a.n_slots = n_blocks * block_size;
    a.n_heads = (uint32_t)n_heads;
    a.block_size = (uint32_t)block_size;
    a.div_block = make_fastdiv((uint32_t)block_size);
    a.qjl_frag = sk->dfrag;
    a.qjl_signs = k_signs;
    a.qjl_gamma = k_gamma;
    if (!tuned_d(pk->d)) {
        // packed rows: block (x, y) = (head, y-th run of g_tpb token tiles)
        if (!packed_decode(pk->d, pk->bits, dtype == ISOQ_F16))
            return ISOQ_E_UNSUPPORTED;
        const void *fn = packed_qjl_kernel_for(pk->variant, pk->d, pk->bits, sk->m, true);
        if (!fn)
            return ISOQ_E_UNSUPPORTED;
        const PackedShape ps = packed_shape(pk->d, pk->bits, true);
        const int64_t per_tile = (int64_t)ps.rows * kPackedQjlWaves * packed_groups(ps.rows, ps.chunks, true);
        const int64_t tiles = (n_tokens + per_tile - 1) / per_tile;
        const int64_t by = std::max<int64_t>(1, std::min<int64_t>(tiles, kQjlBlocks * 4 / kPackedQjlWaves / n_heads));
        const int64_t tpb = (tiles + by - 1) / by;
        const int64_t gy = (tiles + tpb - 1) / tpb;
        if (gy > 65535)
            return ISOQ_E_UNSUPPORTED;
        set_packed_args(pk, ps, tpb, a);
        void *args[] = {&a};
        return launch(fn, dim3((unsigned)n_heads, (unsigned)gy, 1), args, stream, 64 * kPackedQjlWaves);
    }
    const int waves = qjl_waves(sk->m, true, pk->n_sets);
    const void *fn = qjl_kernel_for(pk->variant, pk->d, pk->bits, dtype == ISOQ_F16, sk->m, true, waves);
    if (!fn)
        return ISOQ_E_UNSUPPORTED;
    // block (x, y) = (head, token range); a block stages its head's projection
    // once and walks token ranges y, y + gridDim.y, ... of that head
    const int64_t rpr = rows_per_block(pk) / 4 * waves;   // tokens per range
    const int64_t ranges = (n_tokens + rpr - 1) / rpr;
    const int64_t by = std::max<int64_t>(1, std::min<int64_t>(ranges, kQjlBlocks * 4 / waves / n_heads));
    if (by > 65535)
        return ISOQ_E_UNSUPPORTED;
    void *args[] = {&a};
    return launch(fn, dim3((unsigned)n_heads, (unsigned)by, 1), args, stream, 64 * waves);
}

}  // extern "C"
