// LDS layout of the streamed chunks of the wide matrix-core passes
// (k_mfma_wide.hip, d = 2560).
//
// Plain integer arithmetic, callable from host and device, so that the host
// test tests/test_mfma_layout.py can compile exactly these functions and
// check, on the CPU, that every LDS read returns the element its MFMA
// operand needs.
//
// A wave owns DS columns of the 16 streamed rows of a chunk: G = DS / 8
// granules of 16 bytes per row, rows back to back.  Granule g of row r sits
// at r G + (g ^ (r & 7)) (G is a multiple of 8, so the XOR stays inside the
// row).  Row-wise reads (A operand of the 16x16x32 logit product: lane l
// reads row l % 16, granule 4 kk + l / 16) then put the eight rows a read
// serves together on eight different 16-byte bank groups, and the
// transposing reads of the 16x16x16 second product spread their 8-byte
// pieces over all 64 banks when G = 40.
//
// The chunk reaches LDS from registers: the passes with a second product
// load the logit product's operand straight from the tiled readout copy
// (lane l: row l % 16, granule 4 kk + l / 16 at k-step kk) and write those
// registers to the place a row-wise read of that operand would address
// (rowread_off), where the transposing reads find them.
#pragma once

#if defined(__HIPCC__)
#define SOLO_HDW __host__ __device__ inline
#else
#define SOLO_HDW inline
#endif

namespace solo {
namespace layoutw {

constexpr int NW = 8;   // waves per workgroup
constexpr int YC = 16;  // streamed rows per chunk

template <int DS>
struct Geo {
    static constexpr int G = DS / 8;          // granules per row of a wave slice
    static constexpr int SLOTS = YC * G;      // granules per slice
    static constexpr int SLICE = YC * DS * 2;  // bytes of one wave's chunk slice
    static_assert(G % 8 == 0 && SLOTS % 64 == 0, "slice width: a multiple of 64 columns");
};

// byte offset of granule g (columns 8 g .. 8 g + 7 of the slice) of streamed row r
template <int DS>
SOLO_HDW int phys(int r, int g) {
    return 16 * (r * Geo<DS>::G + (g ^ (r & 7)));
}

// row-wise operand read at k-step kk: lane l, row l % 16, granule 4 kk + l / 16
template <int DS>
SOLO_HDW int rowread_off(int lane, int kk) {
    return phys<DS>(lane & 15, 4 * kk + (lane >> 4));
}

// transposing read (ds_read_b64_tr_b16) for the A operand of the 16x16x16
// second product over column block b (columns 16 b .. 16 b + 15 of the
// slice): lane L of 16-lane group g addresses the 8 bytes of row 4 g + L / 4,
// columns 16 b + 4 (L % 4) .. + 3; lane i of the group then receives, as
// element e, column 16 b + i of row 4 g + e.
template <int DS>
SOLO_HDW int trread_off(int lane, int b) {
    const int g = lane >> 4, L = lane & 15;
    const int row = 4 * g + (L >> 2);
    const int col = 16 * b + 4 * (L & 3);
    return phys<DS>(row, col >> 3) + 2 * (col & 7);
}

}  // namespace layoutw
}  // namespace solo
