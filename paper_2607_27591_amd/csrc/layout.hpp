// Memory layouts of libprox: the packed proxy blob and the workspace.
// Used by both host (api.hip) and device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace prox {

constexpr int kF16 = 0;
constexpr int kBF16 = 1;
constexpr int kMaxDModel = 16384;   // multiple of 128
constexpr int kMaxDFF = 65536;
constexpr int kMaxBatch = 16;

// ---------------------------------------------------------------------------
// Proxy blob
// ---------------------------------------------------------------------------
// [0, 256)           header (BlobHeader)
// codes              for each column tile t (kTile columns of d_ff, the last
//                    tile zero-padded) and each input row i (0..d-1), one
//                    contiguous row segment: kTile gate codes, then kTile up
//                    codes.  INT4: two codes per byte, column 2c in the low
//                    nibble, stored as q + 8 (1..15).  INT8: one byte per
//                    code, stored as q + 128 (1..255).  Input-major, so an
//                    input-sparse proxy reads whole contiguous segments.
// scales (256-aligned) for each tile t and group g: kTile gate scales then
//                    kTile up scales, fp16 bits (0 in padded columns).
constexpr int kTile = 512;              // proxy columns per tile
constexpr uint32_t kBlobMagic = 0x42585250u;  // "PRXB"
constexpr uint32_t kBlobVersion = 1;

struct BlobHeader {
    uint32_t magic, version, fmt, group, d_model, d_ff, tile, qbits;
    uint64_t codes_offset, scales_offset, total_bytes;
};

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct BlobLayout {
    int d, f, qbits, group, n_tiles, f_pad;
    size_t row_bytes;      // bytes of one (tile, row) segment: gate + up
    size_t codes_offset, codes_bytes, scales_offset, scales_bytes, total;
    __host__ __device__ BlobLayout(int d_, int f_, int qbits_, int group_)
        : d(d_), f(f_), qbits(qbits_), group(group_) {
        n_tiles = (f + kTile - 1) / kTile;
        f_pad = n_tiles * kTile;
        row_bytes = (size_t)2 * kTile * qbits / 8;
        codes_offset = 256;
        codes_bytes = (size_t)n_tiles * d * row_bytes;
        scales_offset = align_up(codes_offset + codes_bytes, 256);
        scales_bytes = (size_t)n_tiles * (d / group) * 2 * kTile * sizeof(uint16_t);
        total = align_up(scales_offset + scales_bytes, 256);
    }
};

// ---------------------------------------------------------------------------
// Proxy GEMV decomposition
// ---------------------------------------------------------------------------
constexpr int kProxyRowsPerWave = 64;   // one input row per lane when selecting
constexpr int kProxyWaves = 8;          // waves per workgroup
constexpr int kProxyRowsPerSplit = kProxyRowsPerWave * kProxyWaves;
constexpr int kProxyMaxNB = 4;          // batch rows per proxy launch

// Batch rows a proxy launch is compiled for (1, 2 or 4) given nb <= 4 rows.
__host__ __device__ inline int proxy_nb_t(int nb) { return nb <= 1 ? 1 : nb == 2 ? 2 : 4; }

__host__ __device__ inline int proxy_splits(int d) {
    return (d + kProxyRowsPerSplit - 1) / kProxyRowsPerSplit;
}

// ---------------------------------------------------------------------------
// Stage 2 decomposition
// ---------------------------------------------------------------------------
constexpr int kGateUpMaxNB = 4;         // batch rows per gate/up launch
constexpr int kDownCols = 512;          // output columns per down workgroup
constexpr int kDownWaves = 8;           // waves per down workgroup
constexpr int kDownMaxSplits = 64;      // channel splits of the down projection

// Batch rows a down launch is compiled for (1, 2, 4, 8 or 16); partial sums
// are laid out with this many rows per split.
__host__ __device__ inline int down_nb_t(int nb) {
    return nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : nb <= 8 ? 8 : 16;
}

// ---------------------------------------------------------------------------
// Workspace
// ---------------------------------------------------------------------------
// ctrl (4 KiB): selection results and arrival counters.  The counters are
// cleared by the first kernel of every call, so the workspace needs no
// initialisation by the caller.
struct Ctrl {
    uint32_t in_v, in_cut, ff_v, ff_cut;
    uint32_t pad[60];
    uint32_t proxy_count[512];          // per proxy column tile
    uint32_t down_count[256];           // per down column tile
};
static_assert(sizeof(Ctrl) <= 4096, "ctrl block");

struct WsLayout {
    size_t ctrl, proxy_part, scores, ff_idx, s, down_part, total;
    __host__ __device__ WsLayout(int d, int f, int batch) {
        const int n_tiles = (f + kTile - 1) / kTile;
        const int f_pad = n_tiles * kTile;
        const int nbp = proxy_nb_t(batch < kProxyMaxNB ? batch : kProxyMaxNB);
        size_t o = 0;
        ctrl = o; o += 4096;
        proxy_part = o; o = align_up(o + (size_t)proxy_splits(d) * nbp * 2 * f_pad * 4, 256);
        scores = o; o = align_up(o + (size_t)f_pad * 4, 256);
        ff_idx = o; o = align_up(o + (size_t)f * 4, 256);
        s = o; o = align_up(o + (size_t)batch * f * 4, 256);
        down_part = o; o = align_up(o + (size_t)kDownMaxSplits * down_nb_t(batch) * d * 4, 256);
        total = o;
    }
};

}  // namespace prox
