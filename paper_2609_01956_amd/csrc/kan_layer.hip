// kan_layer.hip -- weight packing, tile planning and launch dispatch of the
// fused KAN-layer forward (eq. kan_forward); the kernels are in
// kan_layer_kernel.h.
#include "kan_layer_kernel.h"

#include <algorithm>
#include <mutex>

#include "kan.h"


namespace kan {

namespace {

using layer_detail::Tr;
using layer_detail::kThreads;

// --------------------------------------------------------------- pack kernel

// One unit of the packed buffer per thread: the kj weights of columns
// [kj * blk, kj * blk + kj) of feature f for output column o, the columns of
// a feature ordered [base_w, coef[.., 0], ..., coef[.., nb - 1]] and
// zero-padded.  With `sparse` (bf16, two blocks per feature) unit blk is
// column half w = blk of feature f, holding columns 4 (e % 4) + 2 w + e / 4,
// and goes to block f % 2 of the pair, half w.  Every unit is one 16-byte
// (bf16) or 8-byte (fp32) store.  Units are numbered in 8 x 8 tiles: eight
// output columns (fastest) by eight consecutive (feature, block) pairs fb =
// f nsb + blk, so a wave stores eight runs of eight consecutive units (whole
// 128-byte lines for bf16) and reads eight coefficient rows over four
// features each.  Units past `units_main` zero the padding blocks of each
// tile.
template <typename T>
__global__ __launch_bounds__(kThreads) void pack_kernel(const T* __restrict__ coef,
                                                        const T* __restrict__ bw,
                                                        T* __restrict__ packed, int in, int out,
                                                        int nb, int nsb, int npairs, int nblk_pad,
                                                        int ntile, int64_t units_main,
                                                        int64_t units, bool sparse) {
    constexpr int KJ = Tr<T>::KJ;
    const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (u >= units) return;
    T v[KJ];
#pragma unroll
    for (int e = 0; e < KJ; ++e) v[e] = T(0);
    int64_t dst;  // unit index in the packed buffer
    if (u < units_main) {
        const int fb_count = 2 * npairs * nsb;
        const int fb_tiles = (fb_count + 7) / 8;
        const int n_lo = (int)(u % 8);
        const int fb_lo = (int)((u / 8) % 8);
        const int64_t w = u / 64;
        const int fb = (int)(w % fb_tiles) * 8 + fb_lo;
        const int o = (int)(w / fb_tiles) * 8 + n_lo;
        if (fb >= fb_count) return;  // (the last (feature, block) tile's padding)
        const int blk = fb % nsb;
        const int f = fb / nsb;
        const int tile = o / ntile, n = o % ntile;
        if (o < out && f < in) {  // (f == in: the phantom feature of an odd count)
            const int64_t row = (int64_t)o * in + f;
#pragma unroll
            for (int e = 0; e < KJ; ++e) {
                const int c = sparse ? 4 * (e % 4) + 2 * blk + e / 4 : blk * KJ + e;
                if (c == 0) v[e] = bw[row];
                else if (c <= nb) v[e] = coef[row * nb + c - 1];
            }
        }
        if (sparse) {
            const int64_t gblk = (int64_t)tile * nblk_pad + (int64_t)(f / 2) * nsb + (f & 1);
            dst = (gblk * 2 + blk) * ntile + n;
        } else {
            const int64_t gblk = (int64_t)tile * nblk_pad + (int64_t)(f / 2) * nsb + blk;
            dst = (gblk * 2 + (f & 1)) * ntile + n;
        }
    } else {
        // padding blocks [npairs * nsb, nblk_pad) of every tile: zeros
        const int64_t q = u - units_main;
        const int64_t per_tile = (int64_t)(nblk_pad - npairs * nsb) * 2 * ntile;
        const int64_t tile = q / per_tile;
        dst = tile * (int64_t)nblk_pad * 2 * ntile + (int64_t)npairs * nsb * 2 * ntile +
              q % per_tile;
    }
    T* d = packed + dst * KJ;
#pragma unroll
    for (int e = 0; e < KJ; ++e) d[e] = v[e];
}

}  // namespace

// ------------------------------------------------------------------ planning

bool layer_geom(int nb, int kdeg, bool bf16, int in, int out, LayerGeom* g) {
    g->nb = nb;
    g->kdeg = kdeg;
    g->out = out;
    g->kj = bf16 ? 8 : 2;
    g->nsb = (nb + 1 + g->kj - 1) / g->kj;
    g->npairs = (in + 1) / 2;
    const int64_t nblk = (int64_t)g->npairs * g->nsb;
    // fp32 tiles are at most 128 columns wide (fp32 MFMA time dwarfs the basis
    // generation, so regenerating it per tile is cheap); bf16 tiles up to 256
    // so each basis value is generated once per row for out <= 256.
    const int nfmax = bf16 ? 8 : 4;
    const int need = (out + 31) / 32;
    int nf = 1;
    while (nf < nfmax && nf < need) nf *= 2;
    g->nf = nf;
    g->ntiles = (out + 32 * nf - 1) / (32 * nf);
    const int64_t blk_bytes = layer_block_bytes(bf16, nf);
    const int kb = layer_chunk_blocks(bf16, nf);
    const int64_t nblk_pad = (nblk + kb - 1) / kb * kb;
    if (nblk_pad > 0x7fffffffLL / 8 || g->ntiles > 65535) return false;
    g->nblk = (int)nblk;
    g->nblk_pad = (int)nblk_pad;
    g->kb = kb;
    // (the structured-sparse operand holds the four nonzero cubic columns)
    g->sparse = bf16 && g->nsb == 2 && kdeg == 3;
    g->packed_bytes = (size_t)g->ntiles * (size_t)nblk_pad * (size_t)blk_bytes;
    return true;
}

bool layer_cfg_valid(const LayerGeom& g, const LayerCfg& c) {
    if (c.rf == 0) return c.wk == 4 && c.nw == 4 && c.cs == 1 && narrow_ok(g);
    // other degrees: the run-time degree build of one shape (one row tile per
    // wave, four waves, whole K and N tile)
    if (g.kdeg != 3) return c.rf == 1 && c.wk == 1 && c.nw == 4 && c.cs == 1;
    // sparse: one row tile per wave, where 256-column tiles take
    // four-wave workgroups only on column slices (the whole 256 columns with
    // four waves' larger share of the weight staging exceed 256 registers
    // and spill), or two row tiles per wave over the whole tile (four waves,
    // or eight on 256-column tiles: column halves sharing A)
    // (sparse K splits: tiles of one or two fragments, one row tile per wave,
    // whole feature pairs per wave slice)
    if (g.sparse && c.wk != 1 &&
        (g.nf > 2 || c.rf != 1 || c.cs != 1 || (g.kb / 2) % c.wk != 0))
        return false;
    if (g.sparse && c.wk == 1 &&
        ((c.rf == 1 && g.nf == 8 && c.nw == 4 && c.cs == 1) || (c.rf == 2 && c.cs != 1)))
        return false;
    // eight waves of two row tiles, or eight waves splitting K: sparse only
    if (!g.sparse && c.nw == 8 && (c.rf == 2 || c.wk != 1)) return false;
    return layer_shape_ok(g.kj == 8, g.nf, c.rf, c.wk, c.nw, c.cs);
}

LayerCfg plan_layer(const LayerGeom& g, bool bf16, int64_t batch) {
    if (g.kdeg != 3) return LayerCfg{1, 1, 4, 1};
    // Narrow fp32 layers on the vector ALUs (kan_narrow.hip) once the batch
    // gives every CU workgroups.
    if (narrow_ok(g) && batch >= 16384) return LayerCfg{0, 4, 4, 1};
    auto wgs = [&](const LayerCfg& c) {
        const int64_t bm = layer_cfg_rows(c);
        return ((batch + bm - 1) / bm) * g.ntiles * c.cs;
    };
    // bf16 with 256-column tiles: 32-row waves (two per SIMD, accumulators in
    // 128 registers) overlap one wave's basis VALU work with the other's MFMAs;
    // 64-row waves (256 accumulator registers) run one wave per SIMD, which
    // measured slower on MI355X.  Eight waves per workgroup halve the weight
    // traffic per row.  Used when it fills the chip (one workgroup per CU).
    const LayerCfg wide{1, 1, 8, 1};
    // On the sparse layout the eight waves take 64 rows each over half the
    // columns instead, passing each other the A of one row tile: the same
    // 256 x 256 workgroup tile, half the LDS bytes of B per MFMA (784 -> 256:
    // 309 us against 329 us).
    const LayerCfg shared_a{2, 1, 8, 1};
    if (bf16 && g.nf == 8 && g.sparse && wgs(shared_a) >= 256) return shared_a;
    if (bf16 && g.nf == 8 && wgs(wide) >= 256) return wide;
    // Sparse layers (bf16, two blocks per feature): one row tile per wave and
    // no K split; eight waves per workgroup when that fills the chip, else
    // four over the whole tile (not for 256-column tiles), else column slices
    // below.  (256 -> 10 at batch 65536: 49 us; 256 -> 100: 73 us with eight
    // waves against 82 us with four.)
    if (g.sparse) {
        // Tiles of one or two fragments: two wave slices splitting the
        // feature pairs (twice the waves for the basis-generation-bound
        // loop; 256 -> 10: 43 us against 46 us, 256 -> 64: 52 against 57).
        const LayerCfg k2{1, 2, 8, 1};
        if (g.nf <= 2 && layer_cfg_valid(g, k2) && wgs(k2) >= 256) return k2;
        const LayerCfg n8{1, 1, 8, 1}, n4{1, 1, 4, 1};
        if (wgs(n8) >= 256) return n8;
        if (layer_cfg_valid(g, n4) && wgs(n4) >= 256) return n4;
    }
    // Otherwise the tallest workgroup over the whole N tile (fewest re-reads
    // of the weights, basis values generated once per tile) that still gives
    // at least `want` workgroups; the basis-generation-bound narrow layers
    // (one 32-column fragment) want more, smaller workgroups.  Splitting the tile's columns over
    // 2 or 4 workgroups (each stages only its columns and regenerates the
    // basis) measured slower whenever every CU already had a workgroup, so it
    // is taken only for batches too small for that.
    const int64_t want = g.nf == 1 ? 1024 : 512;
    const LayerCfg whole[] = {{2, 1, 4, 1}, {1, 1, 4, 1}, {1, 2, 4, 1}, {1, 4, 4, 1}};
    const LayerCfg sliced[] = {{1, 1, 4, 2}, {1, 2, 4, 2}, {1, 4, 4, 2},
                               {1, 1, 4, 4}, {1, 2, 4, 4}, {1, 4, 4, 4}};
    LayerCfg best{1, 1, 4, 1};
    int64_t best_wgs = 0;
    for (const LayerCfg& c : whole) {
        if (!layer_cfg_valid(g, c)) continue;
        const int64_t w = wgs(c);
        if (w >= want) return c;
        // (on a tie, the later shape: fewer rows per workgroup, more waves on K)
        if (w >= best_wgs) { best = c; best_wgs = w; }
    }
    if (best_wgs >= 256) return best;
    for (const LayerCfg& c : sliced) {
        if (!layer_cfg_valid(g, c)) continue;
        const int64_t w = wgs(c);
        if (w > best_wgs) { best = c; best_wgs = w; }
        if (w >= 256) return c;
    }
    return best;  // the most workgroups any shape gives
}

// ----------------------------------------------------- no-allocation scratch

namespace {

// Packed weights of kan_layer_forward_noalloc.  Each GPU the library runs on
// holds its own copy for the life of the process.  In host code `scratch`
// names a host-side stand-in, not device memory: kernels only ever receive
// the device address from hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[KAN_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_addr[kMaxDevices];

}  // namespace

hipError_t noalloc_scratch(void** ptr, size_t* bytes) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (scratch_addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        scratch_addr[dev] = p;
    }
    *ptr = scratch_addr[dev];
    *bytes = KAN_NOALLOC_SCRATCH_BYTES;
    return hipSuccess;
}

// ------------------------------------------------------------------ launches

hipError_t launch_pack(bool bf16, const LayerGeom& g, int in, int out, const void* coef,
                       const void* base_w, void* packed, hipStream_t s) {
    const int ntile = 32 * g.nf;
    // (feature, block) pairs rounded up to whole tiles of eight (pack_kernel)
    const int64_t units_main = (int64_t)g.ntiles * ntile * ((2 * g.npairs * g.nsb + 7) / 8 * 8);
    const int64_t units =
        units_main + (int64_t)g.ntiles * (g.nblk_pad - g.npairs * g.nsb) * 2 * ntile;
    const unsigned blocks = (unsigned)((units + kThreads - 1) / kThreads);
    if (bf16)
        hipLaunchKernelGGL(pack_kernel<uint16_t>, dim3(blocks), dim3(kThreads), 0, s,
                           static_cast<const uint16_t*>(coef),
                           static_cast<const uint16_t*>(base_w), static_cast<uint16_t*>(packed),
                           in, out, g.nb, g.nsb, g.npairs, g.nblk_pad, ntile, units_main, units,
                           g.sparse);
    else
        hipLaunchKernelGGL(pack_kernel<float>, dim3(blocks), dim3(kThreads), 0, s,
                           static_cast<const float*>(coef), static_cast<const float*>(base_w),
                           static_cast<float*>(packed), in, out, g.nb, g.nsb, g.npairs,
                           g.nblk_pad, ntile, units_main, units, false);
    return hipGetLastError();
}

namespace {

// y = sum over the K splits of the partial sums, in split order.  The loads
// go out 16 at a time before their adds, so a small batch (one workgroup
// reading many splits) waits on one memory round trip per 16 splits rather
// than one per split.  The +0 that stands in for a split past the last one
// leaves the sum bitwise unchanged (the sum starts at +0 and never becomes
// -0).
template <typename T>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ P,
                                                           T* __restrict__ y, int64_t n, int ks) {
    constexpr int kBatch = 16;
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= n) return;
    float v = 0.0f;
    for (int z0 = 0; z0 < ks; z0 += kBatch) {
        float t[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i)
            t[i] = z0 + i < ks ? P[(int64_t)(z0 + i) * n + u] : 0.0f;
#pragma unroll
        for (int i = 0; i < kBatch; ++i) v += t[i];
    }
    if constexpr (sizeof(T) == 2) y[u] = f32_to_bf16(v);
    else y[u] = v;
}

int layer_chunks(const LayerGeom& g) { return g.nblk_pad / g.kb; }

}  // namespace

int layer_k_splits(const LayerGeom& g, const LayerCfg& c, int64_t batch, int out) {
    // Split only where the workgroups give fewer than two per CU, towards
    // kSplitTargetWgs workgroups (fp32 shapes hold fewer registers and more
    // workgroups per CU than bf16 ones), never into splits of fewer than 4
    // chunks and 16 blocks (pipeline fill and drain; the 256-column bf16
    // tiles have 2 blocks per chunk, the others 8), and with at most
    // kSplitMaxPartialBytes of partial sums (written and read back once
    // more).  Measured on MI355X at batches 1 to 4096 of 784 -> 64, 784 ->
    // 256, 256 -> 256 and 256 -> 10 layers in both dtypes.
    constexpr int64_t kSplitBelowWgs = 512;
    const int64_t kSplitTargetWgs = g.kj == 8 ? 512 : 2048;
    const int kSplitMinChunks = std::max(4, 16 / g.kb);
    constexpr int64_t kSplitMaxPartialBytes = (int64_t)16 << 20;
    const int64_t bm = layer_cfg_rows(c);
    const int64_t wgs = ((batch + bm - 1) / bm) * g.ntiles * c.cs;
    const int nch = layer_chunks(g);
    // (the narrow-layer kernel and the shared-A shape, whose epilogue stores
    // bf16 rows through LDS, never split)
    if (c.rf == 0 || (c.rf == 2 && c.nw == 8) || nch < 2 * kSplitMinChunks ||
        wgs >= kSplitBelowWgs)
        return 1;
    int64_t ks = (kSplitTargetWgs + wgs - 1) / wgs;
    ks = std::min<int64_t>(ks, nch / kSplitMinChunks);
    ks = std::min<int64_t>(ks, kSplitMaxPartialBytes / (batch * (int64_t)out * 4));
    if (ks <= 1) return 1;
    const int cps = (int)((nch + ks - 1) / ks);
    return (nch + cps - 1) / cps;
}

size_t layer_partial_bytes(const LayerGeom& g, const LayerCfg& c, int64_t batch, int out) {
    const int ks = layer_k_splits(g, c, batch, out);
    if (ks <= 1) return 0;
    return ((size_t)ks * (size_t)batch * (size_t)out * 4 + 255) & ~(size_t)255;
}

hipError_t launch_layer(bool bf16, const LayerGeom& g, const LayerCfg& c, LayerArgs a, int ks,
                        void* partial, hipStream_t s) {
    if (!layer_cfg_valid(g, c)) return hipErrorInvalidValue;
    if (c.rf == 0) return ks == 1 ? launch_narrow(g, a, s) : hipErrorInvalidValue;
    const int nch = layer_chunks(g);
    if (ks < 1 || ks > nch || (ks > 1 && partial == nullptr)) return hipErrorInvalidValue;
    a.cps = (nch + ks - 1) / ks;
    ks = (nch + a.cps - 1) / a.cps;
    a.P = ks > 1 ? static_cast<float*>(partial) : nullptr;
    hipError_t e = bf16 ? launch_layer_bf16(g, c, a, s) : launch_layer_f32(g, c, a, s);
    if (e != hipSuccess || ks == 1) return e;
    const int64_t n = a.batch * (int64_t)a.out;
    const unsigned blocks = (unsigned)((n + 255) / 256);
    if (bf16)
        hipLaunchKernelGGL(split_reduce_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s,
                           a.P, static_cast<uint16_t*>(a.y), n, ks);
    else
        hipLaunchKernelGGL(split_reduce_kernel<float>, dim3(blocks), dim3(256), 0, s, a.P,
                           static_cast<float*>(a.y), n, ks);
    return hipGetLastError();
}

}  // namespace kan
