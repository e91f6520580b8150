// Memory layouts of libprox: the packed proxy blob, the launch geometry of
// the three kernels, and the workspace.  Used by host and device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace prox {

constexpr int kF16 = 0;
constexpr int kBF16 = 1;
constexpr int kMaxDModel = 16384;   // multiple of 128
constexpr int kMaxDFF = 65536;
constexpr int kBlock = 1024;        // threads per workgroup of the main kernels
constexpr int kMaxBlockWaves = kBlock / 64;

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// Proxy blob
// ---------------------------------------------------------------------------
// [0, 256)            header (BlobHeader)
// codes               for each input row i (0..d-1) and each column tile t
//                     (T columns of d_ff; the last tile zero-padded), one
//                     contiguous segment: T gate codes then T up codes.
//                     INT4: two codes per byte, even column in the low nibble,
//                     stored as q + 8 (1..15).  INT8: one byte, q + 128.
//                     Row-major over tiles: the segments of one kept input row
//                     for all tiles are one contiguous run, and the workgroups
//                     (one per tile) walk the same kept-row list in step, so
//                     the input-sparse proxy GEMV reaches DRAM as long runs.
// scales (256-aligned) for each tile t and group g: T gate scales then T up
//                     scales, fp16 bits (0 in padded columns).
// The tile width T is 128 when that already gives kProxyMinTiles column tiles
// (one workgroup each), else 64.
constexpr int kProxyMinTiles = 192;
constexpr uint32_t kBlobMagic = 0x42585250u;  // "PRXB"
constexpr uint32_t kBlobVersion = 3;

__host__ __device__ inline int proxy_tile(int f) {
    return (f + 127) / 128 >= kProxyMinTiles ? 128 : 64;
}

struct BlobHeader {
    uint32_t magic, version, fmt, group, d_model, d_ff, tile, qbits;
    uint64_t codes_offset, scales_offset, total_bytes;
};

struct BlobLayout {
    int d, f, qbits, group, tile, n_tiles, f_pad;
    size_t row_bytes;      // bytes of one (row, tile) segment: gate + up
    size_t row_stride;     // bytes between the segments of rows i and i + 1
    size_t codes_offset, codes_bytes, scales_offset, scales_bytes, total;
    __host__ __device__ BlobLayout(int d_, int f_, int qbits_, int group_)
        : d(d_), f(f_), qbits(qbits_), group(group_) {
        tile = proxy_tile(f);
        n_tiles = (f + tile - 1) / tile;
        f_pad = n_tiles * tile;
        row_bytes = (size_t)2 * tile * qbits / 8;
        row_stride = (size_t)n_tiles * row_bytes;
        codes_offset = 256;
        codes_bytes = (size_t)d * row_stride;
        scales_offset = align_up(codes_offset + codes_bytes, 256);
        scales_bytes = (size_t)n_tiles * (d / group) * 2 * tile * sizeof(uint16_t);
        total = align_up(scales_offset + scales_bytes, 256);
    }
};

// ---------------------------------------------------------------------------
// Stage 1: proxy GEMV + score, one workgroup per column tile.
// ---------------------------------------------------------------------------
constexpr int kProxyMaxNB = 4;           // batch rows per proxy launch

__host__ __device__ inline int proxy_nb_t(int nb) { return nb <= 1 ? 1 : nb == 2 ? 2 : 4; }

// ---------------------------------------------------------------------------
// Stage 2: fused channel select + gate/up + down.  Each workgroup takes an
// equal slice of the kept channels and writes one partial y.
// ---------------------------------------------------------------------------
constexpr int kStage2MaxWGs = 256;
constexpr int kStage2MinChannels = 8;    // per workgroup, before shrinking the grid

__host__ __device__ inline int stage2_wgs(int n_ch) {
    int w = (n_ch + kStage2MinChannels - 1) / kStage2MinChannels;
    return w < 1 ? 1 : (w > kStage2MaxWGs ? kStage2MaxWGs : w);
}

// INT4 base weights for Stage 2 (W4A16).  For each matrix m (gate, up, down),
// channel-major codes [f][d/2] (column i of row j in byte i/2: the low nibble
// when i is even, as q + 8) and fp16 scales [f][d/group]; every array starts
// on a 256-byte boundary.
struct W4Layout {
    size_t codes[3], scales[3], total;
    __host__ __device__ W4Layout(int d, int f, int group) {
        size_t off = 0;
        for (int m = 0; m < 3; ++m) {
            codes[m] = off;
            off = align_up(off + (size_t)f * (size_t)(d / 2), 256);
        }
        for (int m = 0; m < 3; ++m) {
            scales[m] = off;
            off = align_up(off + (size_t)f * (size_t)(d / group) * 2, 256);
        }
        total = off;
    }
};

constexpr int kStage2MaxNB = 8;          // batch rows per Stage 2 launch
constexpr int kStage2MfmaRows = 16;      // ... of the matrix-core Stage 2 (16-bit weights)
constexpr int kStage2DownGroups = 64;    // kept-channel groups of its down projection

// Batch rows a Stage 2 launch of nb <= 8 rows is compiled for (1, 2, 4 or 8).
__host__ __device__ inline int stage2_nb_t(int nb) {
    return nb <= 1 ? 1 : nb <= 2 ? 2 : nb <= 4 ? 4 : 8;
}

// Rows of partial y each Stage 2 workgroup owns in the workspace for a batch.
__host__ __device__ inline int ypart_rows(int batch) {
    return batch <= kStage2MaxNB ? stage2_nb_t(batch)
                                 : (batch + kStage2MaxNB - 1) / kStage2MaxNB * kStage2MaxNB;
}

// How a launch selects its set (Sec. 4.1 masks): by count (the top-k reading,
// App. A.6) or, with tau_mode, by the layer-wise threshold rule |z| >= tau,
// whose realised count then goes to *count (when count is not NULL).
struct Select {
    int tau_mode;
    float tau;
    int32_t *count;
};

// ---------------------------------------------------------------------------
// Workspace (no initialisation needed)
// ---------------------------------------------------------------------------
// scores: the proxy scores (fp32, f padded to 128); ypart: the partial y rows
// of Stage 2, one set per Stage 2 workgroup (kStage2MaxWGs), or per
// kept-channel group of the matrix-core down projection (kStage2DownGroups)
// when a batch of more than kStage2MaxNB rows of 16-bit weights takes that
// path; sbuf (that path only): s of the kept channels in kept-list order,
// [f][kStage2MfmaRows] fp32.  wq: 16 for 16-bit weights, 4 for INT4 ones.
// Shapes the matrix-core Stage 2 takes: 16-bit weights, d_model >= 4096.
__host__ __device__ inline bool stage2_mfma_shape(int d, int wq) { return wq == 16 && d >= 4096; }
__host__ __device__ inline bool ws_mfma_path(int d, int batch, int wq) {
    return batch > kStage2MaxNB && stage2_mfma_shape(d, wq);
}
struct WsLayout {
    size_t scores, klist, ypart, sbuf, total;
    __host__ __device__ WsLayout(int d, int f, int batch, int wq) {
        const int f_pad = (f + 127) / 128 * 128;
        const bool mfma = ws_mfma_path(d, batch, wq);
        const size_t groups = mfma ? kStage2DownGroups : kStage2MaxWGs;
        size_t o = 0;
        scores = o; o = align_up(o + (size_t)f_pad * 4, 256);
        klist = o; o = align_up(o + (size_t)(f + 1) * 4, 256);   // kept channels, then their count
        ypart = o; o = align_up(o + groups * ypart_rows(batch) * d * 4, 256);
        sbuf = o;
        if (mfma) o = align_up(o + (size_t)f * kStage2MfmaRows * 4, 256);
        total = o;
    }
};

}  // namespace prox
