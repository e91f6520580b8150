// Proxy packing (Sec. 4.3): symmetric per-(channel, group) quantisation of
// W_gate and W_up into the tiled, input-major proxy blob, and the inverse
// view used for inspection.
#include "common.hpp"
#include "kernels.hpp"

namespace prox {

// IEEE binary16 round-to-nearest-even of a binary64 value, from the bit
// fields of the double.
__device__ uint16_t f64_to_f16_rne(double v) {
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint16_t sign = (uint16_t)((u >> 48) & 0x8000u);
    const uint64_t a = u & 0x7FFFFFFFFFFFFFFFull;
    if (a >= 0x7FF0000000000000ull) return sign | (a > 0x7FF0000000000000ull ? 0x7E00 : 0x7C00);
    if (a < 0x0010000000000000ull) return sign;   // below 2^-1022: rounds to zero
    const int e = (int)(a >> 52) - 1023;
    if (e > 15) return sign | 0x7C00;
    const uint64_t m = (a & 0x000FFFFFFFFFFFFFull) | 0x0010000000000000ull;  // 53 bits
    // Normal results keep 11 significant bits; subnormal ones count 2^-24 units.
    const int shift = e >= -14 ? 42 : 28 - e;
    if (shift > 62) return sign;
    uint64_t keep = m >> shift;
    const uint64_t rem = m & ((1ull << shift) - 1);
    const uint64_t half = 1ull << (shift - 1);
    if (rem > half || (rem == half && (keep & 1))) ++keep;
    if (e >= -14) {
        int E = e;
        if (keep == 2048) { keep = 1024; ++E; }
        if (E > 15) return sign | 0x7C00;
        return sign | (uint16_t)((E + 15) << 10) | (uint16_t)(keep - 1024);
    }
    return sign | (uint16_t)keep;   // 1024 encodes the smallest normal
}

__device__ __forceinline__ double f16_to_f64(uint16_t h) {
    return (double)f16_bits_to_float(h);
}

template <int DT>
__device__ __forceinline__ double w_to_f64(uint16_t h) { return (double)half_to_float<DT>(h); }

// One thread per (matrix, group, column pair).  Two adjacent columns share an
// INT4 byte, so a thread owns both.
template <int DT, int QB>
__global__ __launch_bounds__(256) void pack_kernel(const uint16_t *__restrict__ wg,
                                                   const uint16_t *__restrict__ wu, int d, int f,
                                                   int group, uint8_t *__restrict__ blob) {
    const BlobLayout L(d, f, QB, group);
    const int ng = d / group;
    const int npairs = L.f_pad / 2;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid == 0) {
        BlobHeader h{};
        h.magic = kBlobMagic; h.version = kBlobVersion; h.fmt = QB == 4 ? 1u : QB == 8 ? 0u : 2u;
        h.group = (uint32_t)group; h.d_model = (uint32_t)d; h.d_ff = (uint32_t)f;
        h.tile = (uint32_t)L.tile; h.qbits = QB;
        h.codes_offset = L.codes_offset; h.scales_offset = L.scales_offset;
        h.total_bytes = L.total;
        *reinterpret_cast<BlobHeader *>(blob) = h;
    }
    if (gid >= 2LL * ng * npairs) return;
    const int mat = (int)(gid / ((long long)ng * npairs));
    const int rem = (int)(gid % ((long long)ng * npairs));
    const int g = rem / npairs;
    const int j0 = (rem % npairs) * 2;
    const uint16_t *w = mat == 0 ? wg : wu;
    constexpr int qmax = QB == 4 ? 7 : 127;
    const int T = L.tile;
    const int tile = j0 / T, c0 = j0 % T;
    if constexpr (QB == 16) {
        // Unquantised proxy: the weights' own 16-bit patterns, unit scales.
        uint16_t *scales = reinterpret_cast<uint16_t *>(blob + L.scales_offset);
        const size_t sb = (((size_t)tile * ng + g) * 2 + mat) * T + c0;
        scales[sb] = 0x3C00u;   // fp16 1.0
        scales[sb + 1] = 0x3C00u;
        for (int ii = 0; ii < group; ++ii) {
            const int i = g * group + ii;
            uint16_t *seg = reinterpret_cast<uint16_t *>(blob + L.codes_offset + (size_t)i * L.row_stride +
                                                         (size_t)tile * L.row_bytes);
            seg[mat * T + c0] = j0 < f ? w[(size_t)j0 * d + i] : (uint16_t)0;
            seg[mat * T + c0 + 1] = j0 + 1 < f ? w[(size_t)(j0 + 1) * d + i] : (uint16_t)0;
        }
        return;
    }

    double sigma[2];
    uint16_t sbits[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int j = j0 + e;
        double amax = 0.0;
        if (j < f) {
            const uint16_t *row = w + (size_t)j * d + (size_t)g * group;
            for (int i = 0; i < group; ++i) amax = fmax(amax, fabs(w_to_f64<DT>(row[i])));
        }
        sbits[e] = f64_to_f16_rne(amax / (double)qmax);
        sigma[e] = f16_to_f64(sbits[e]);
    }
    uint16_t *scales = reinterpret_cast<uint16_t *>(blob + L.scales_offset);
    const size_t sbase = (((size_t)tile * ng + g) * 2 + mat) * T + c0;
    scales[sbase] = sbits[0];
    scales[sbase + 1] = sbits[1];

    uint8_t *codes = blob + L.codes_offset;
    for (int ii = 0; ii < group; ++ii) {
        const int i = g * group + ii;
        int q[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int j = j0 + e;
            q[e] = 0;
            if (j < f && sigma[e] != 0.0) {
                double r = rint(w_to_f64<DT>(w[(size_t)j * d + i]) / sigma[e]);
                r = fmin(fmax(r, (double)-qmax), (double)qmax);
                q[e] = (int)r;
            }
        }
        uint8_t *seg = codes + (size_t)i * L.row_stride + (size_t)tile * L.row_bytes;
        if constexpr (QB == 4) {
            seg[mat * (T / 2) + c0 / 2] = (uint8_t)((q[0] + 8) | ((q[1] + 8) << 4));
        } else {
            seg[mat * T + c0] = (uint8_t)(q[0] + 128);
            seg[mat * T + c0 + 1] = (uint8_t)(q[1] + 128);
        }
    }
}

// Inverse view: one thread per (matrix, channel, group).
template <int QB>
__global__ __launch_bounds__(256) void unpack_kernel(const uint8_t *__restrict__ blob, int d,
                                                     int f, int group, int8_t *cg, uint16_t *sg,
                                                     int8_t *cu, uint16_t *su) {
    const BlobLayout L(d, f, QB, group);
    const int ng = d / group;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= 2LL * f * ng) return;
    const int mat = (int)(gid / ((long long)f * ng));
    const int rem = (int)(gid % ((long long)f * ng));
    const int j = rem / ng, g = rem % ng;
    const int T = L.tile;
    const int tile = j / T, c = j % T;
    const uint16_t *scales = reinterpret_cast<const uint16_t *>(blob + L.scales_offset);
    (mat == 0 ? sg : su)[(size_t)j * ng + g] = scales[(((size_t)tile * ng + g) * 2 + mat) * T + c];
    int8_t *out = (mat == 0 ? cg : cu) + (size_t)j * d;
    for (int ii = 0; ii < group; ++ii) {
        const int i = g * group + ii;
        const uint8_t *seg = blob + L.codes_offset + (size_t)i * L.row_stride + (size_t)tile * L.row_bytes;
        int q;
        if constexpr (QB == 4) {
            const uint8_t byte = seg[mat * (T / 2) + c / 2];
            q = (int)((c & 1) ? (byte >> 4) : (byte & 15)) - 8;
        } else {
            q = (int)seg[mat * T + c] - 128;
        }
        out[i] = (int8_t)q;
    }
}

// INT4 base weights (W4A16): one thread per (matrix, channel, group), the
// same symmetric quantiser as the proxy (scale = amax / 7 rounded to fp16,
// q = round-half-even of w / scale in fp64, clamped to +-7), stored
// channel-major.
template <int DT>
__global__ __launch_bounds__(256) void pack_w4_kernel(const uint16_t *__restrict__ wg,
                                                      const uint16_t *__restrict__ wu,
                                                      const uint16_t *__restrict__ wd, int d, int f,
                                                      int group, uint8_t *__restrict__ blob) {
    const W4Layout L(d, f, group);
    const int ng = d / group;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= 3LL * f * ng) return;
    const int m = (int)(gid / ((long long)f * ng));
    const int rem = (int)(gid % ((long long)f * ng));
    const int j = rem / ng, g = rem % ng;
    const uint16_t *w = (m == 0 ? wg : m == 1 ? wu : wd) + (size_t)j * d + (size_t)g * group;
    double amax = 0.0;
    for (int i = 0; i < group; ++i) amax = fmax(amax, fabs(w_to_f64<DT>(w[i])));
    const uint16_t sbits = f64_to_f16_rne(amax / 7.0);
    const double sigma = f16_to_f64(sbits);
    reinterpret_cast<uint16_t *>(blob + L.scales[m])[(size_t)j * ng + g] = sbits;
    uint8_t *codes = blob + L.codes[m] + (size_t)j * (d / 2) + (size_t)g * (group / 2);
    for (int i = 0; i < group; i += 2) {
        int q[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            q[e] = 0;
            if (sigma != 0.0) {
                const double r = rint(w_to_f64<DT>(w[i + e]) / sigma);
                q[e] = (int)fmin(fmax(r, -7.0), 7.0);
            }
        }
        codes[i / 2] = (uint8_t)((q[0] + 8) | ((q[1] + 8) << 4));
    }
}

// Inverse view of matrix m: codes int8 [f][d] and scales [f][d/group].
__global__ __launch_bounds__(256) void unpack_w4_kernel(const uint8_t *__restrict__ blob, int d,
                                                        int f, int group, int m, int8_t *codes,
                                                        uint16_t *scales) {
    const W4Layout L(d, f, group);
    const int ng = d / group;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long long)f * ng) return;
    const int j = (int)(gid / ng), g = (int)(gid % ng);
    scales[(size_t)j * ng + g] =
        reinterpret_cast<const uint16_t *>(blob + L.scales[m])[(size_t)j * ng + g];
    const uint8_t *src = blob + L.codes[m] + (size_t)j * (d / 2) + (size_t)g * (group / 2);
    int8_t *out = codes + (size_t)j * d + (size_t)g * group;
    for (int i = 0; i < group; i += 2) {
        const uint8_t byte = src[i / 2];
        out[i] = (int8_t)((int)(byte & 15) - 8);
        out[i + 1] = (int8_t)((int)(byte >> 4) - 8);
    }
}

hipError_t launch_pack_w4(int dtype, const void *wg, const void *wu, const void *wd, int d, int f,
                          int group, void *blob, hipStream_t s) {
    const long long n = 3LL * f * (d / group);
    const int nb = (int)((n + 255) / 256);
    auto *g = static_cast<const uint16_t *>(wg);
    auto *u = static_cast<const uint16_t *>(wu);
    auto *dn = static_cast<const uint16_t *>(wd);
    auto *b = static_cast<uint8_t *>(blob);
    if (dtype == kBF16) pack_w4_kernel<kBF16><<<nb, 256, 0, s>>>(g, u, dn, d, f, group, b);
    else pack_w4_kernel<kF16><<<nb, 256, 0, s>>>(g, u, dn, d, f, group, b);
    return hipGetLastError();
}

hipError_t launch_unpack_w4(const void *blob, int d, int f, int group, int m, int8_t *codes,
                            uint16_t *scales, hipStream_t s) {
    const long long n = (long long)f * (d / group);
    const int nb = (int)((n + 255) / 256);
    unpack_w4_kernel<<<nb, 256, 0, s>>>(static_cast<const uint8_t *>(blob), d, f, group, m,
                                        codes, scales);
    return hipGetLastError();
}

hipError_t launch_pack(int dtype, int qbits, const void *wg, const void *wu, int d, int f,
                       int group, void *blob, hipStream_t s) {
    const BlobLayout L(d, f, qbits, group);
    const long long n = 2LL * (d / group) * (L.f_pad / 2);
    const int nb = (int)((n + 255) / 256);
    auto *g = static_cast<const uint16_t *>(wg);
    auto *u = static_cast<const uint16_t *>(wu);
    auto *b = static_cast<uint8_t *>(blob);
    if (dtype == kBF16 && qbits == 4) pack_kernel<kBF16, 4><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    else if (dtype == kBF16 && qbits == 8) pack_kernel<kBF16, 8><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    else if (dtype == kBF16) pack_kernel<kBF16, 16><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    else if (qbits == 4) pack_kernel<kF16, 4><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    else if (qbits == 8) pack_kernel<kF16, 8><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    else pack_kernel<kF16, 16><<<nb, 256, 0, s>>>(g, u, d, f, group, b);
    return hipGetLastError();
}

hipError_t launch_unpack(int qbits, const void *blob, int d, int f, int group, int8_t *cg,
                         uint16_t *sg, int8_t *cu, uint16_t *su, hipStream_t s) {
    const long long n = 2LL * f * (d / group);
    const int nb = (int)((n + 255) / 256);
    auto *b = static_cast<const uint8_t *>(blob);
    if (qbits == 4) unpack_kernel<4><<<nb, 256, 0, s>>>(b, d, f, group, cg, sg, cu, su);
    else unpack_kernel<8><<<nb, 256, 0, s>>>(b, d, f, group, cg, sg, cu, su);
    return hipGetLastError();
}

}  // namespace prox
