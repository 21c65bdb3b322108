// LDS layout of the streamed chunks of the matrix-core passes with a second
// product (k_mfma.hip), and the tiled copy the other passes stream.
//
// Plain integer arithmetic, callable from host and device, so that the host
// test tests/test_mfma_layout.py can compile exactly these functions and
// check, on the CPU, that every LDS read returns the element the MFMA
// operand needs.
#pragma once

#if defined(__HIPCC__)
#define SOLO_HD __host__ __device__ inline
#else
#define SOLO_HD inline
#endif

namespace solo {
namespace layout {

constexpr int NW = 8;   // waves per workgroup of the two-waves-per-SIMD kernels
constexpr int YC = 16;  // streamed rows per chunk

template <int DS>
struct Geo {
    // wave w owns columns [w DS, (w + 1) DS) of the streamed rows
    static constexpr int GPR = DS / 8;                      // 16-byte granules per row of a wave slice
    static constexpr int NI = DS / 32;                      // 1 KiB direct-to-LDS instructions per slice
    // padded layout (DS = 128, 256, 512): every 1 KiB instruction covers whole rows
    static constexpr bool PADDED = (NI % 4) == 0 && (512 % DS) == 0;
    static constexpr int IPITCH = PADDED ? 1088 : 1024;     // bytes between the instructions' destinations
    static constexpr int SLICE = (NI - 1) * IPITCH + 1024;  // bytes of one wave's chunk slice
    // XOR key of the padded layout: (r >> KS) & 3 (see phys).  KS = 1 makes
    // both reads conflict-free under the bank model; measured 2% faster than
    // KS = 2 at DS = 256 and 3% faster at DS = 128
    static constexpr int KS = 1;
    static constexpr int NV = PADDED ? (NI >> KS) : NI;     // distinct per-lane stream offsets
    static_assert(DS % 32 == 0 && DS >= 32 && DS <= 512, "slice width");
};

// Tiled copy of a streamed matrix (the layout tiled_elems sizes), streamed by
// the passes that read their operand straight into registers: 16-byte
// granule o of chunk c holds row 16 c + tile_row(o), columns tile_col(o) ..
// tile_col(o) + 7.  A wave that loads 16 bytes per lane at granule 64 b + lane
// receives the A operand of a 16x16x32 MFMA over columns 32 b .. 32 b + 31
// (row lane % 16, columns 32 b + 8 (lane / 16) .. + 7).
SOLO_HD int tile_row(int o) { return o & 15; }
SOLO_HD int tile_col(int o) { return 32 * (o >> 6) + 8 * ((o & 63) >> 4); }

// Byte offset of 16-byte granule g (columns 8 g .. 8 g + 7 of the slice) of
// streamed row r (0..15) inside a wave's chunk slice.
//
// Padded layout: instruction q of the direct-to-LDS stream writes rows
// q, q + NI, ... (one row if DS = 512) back to back at q * 1088 (so its rows
// start at byte 64 q mod 256); inside a row, the low two bits of the granule
// index are XORed with (r >> KS) & 3.  Under the LDS service model measured on
// gfx950 (a 16-byte-per-lane read served 8 lanes over 32 banks per pass, the
// 8-byte transposing read 32 lanes over 64 banks) the transposing reads (4
// rows x 4 granules) are conflict-free with KS = 1 or 2; with KS = 1 the
// row-wise reads (16 rows at one granule) are too (rows r and r + 1 differ in
// the start bank of their instruction, pairs of rows in the XOR key), with
// KS = 2 they would be 2-way.  The offset stays additive in g >> 2, so
// unrolled loops address with immediates.
// Linear layout (other widths): rows back to back.
template <int DS>
SOLO_HD int phys(int r, int g) {
    using G = Geo<DS>;
    if constexpr (G::PADDED) {
        const int q = r % G::NI, k = r / G::NI;
        return q * G::IPITCH + k * (DS * 2) + 16 * (4 * (g >> 2) + ((g & 3) ^ ((r >> G::KS) & 3)));
    } else {
        return (r * G::GPR + g) * 16;
    }
}

// Direct-to-LDS stream of one chunk: instruction q writes 16 bytes per lane at
// slice + stream_lds_off(q) + 16 lane, fetched from the element offset
// stream_row0(q) * d + stream_voff(...) / 2 relative to the chunk's first row.
template <int DS>
SOLO_HD int stream_lds_off(int q) {
    return q * Geo<DS>::IPITCH;
}

template <int DS>
SOLO_HD int stream_row0(int q) {
    return Geo<DS>::PADDED ? q : 0;
}

// Which per-lane offset register instruction q uses.
template <int DS>
SOLO_HD int stream_vidx(int q) {
    return Geo<DS>::PADDED ? (q >> Geo<DS>::KS) : q;
}

// Per-lane byte offset for offset register v (0 .. NV-1), width d, slice start js.
// Padded: instruction q fetches rows q + NI k (k = lane / GPR); the offset
// depends on q only through q >> KS (NI is a multiple of 4, so (r >> KS) & 3
// of row q + NI k is ((q >> KS) + (NI >> KS) k) & 3).
template <int DS>
SOLO_HD int stream_voff(int v, int d, int js, int lane) {
    using G = Geo<DS>;
    if constexpr (G::PADDED) {
        const int k = lane / G::GPR, s = lane % G::GPR;
        const int x = (v + (G::NI >> G::KS) * k) & 3;  // (r >> KS) & 3 of row r = q + NI k with q >> KS = v
        const int g = 4 * (s >> 2) + ((s & 3) ^ x);
        return (G::NI * k * d + js + 8 * g) * 2;
    } else {
        const int lin = v * 64 + lane;
        const int r = lin / G::GPR, g = lin % G::GPR;
        return (r * d + js + 8 * g) * 2;
    }
}

// Row-wise operand reads (A of the 16x16x32 logit product): lane reads row
// lane % 16, columns 32 kk + 8 (lane / 16) .. +7 at rowread_off(lane) + 64 kk.
template <int DS>
SOLO_HD int rowread_off(int lane) {
    return phys<DS>(lane & 15, lane >> 4);
}

// Transposing operand reads (A of the 32x32x16 second product), one
// ds_read_b64_tr_b16 each for rows 8 hh + 4 half + (0..3) of 32-column block
// b at trread_off(lane, half) + 64 b: lane (16-lane group tg, index ti)
// addresses row 8 (tg / 2) + 4 half + ti / 4, columns 16 (tg % 2) + 4 (ti % 4) .. +3.
template <int DS>
SOLO_HD int trread_off(int lane, int half) {
    const int tg = lane >> 4, ti = lane & 15;
    const int row = 8 * (tg >> 1) + 4 * half + (ti >> 2);
    const int gran = 2 * (tg & 1) + ((ti & 3) >> 1);
    return phys<DS>(row, gran) + ((ti & 1) << 3);
}

}  // namespace layout
}  // namespace solo
