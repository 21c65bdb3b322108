// Host check of the data layouts of the matrix-core passes, with the same
// headers the kernels include:
//   - 16-row tiling, passes with a second product: emulate the direct-to-LDS
//     stream of one chunk slice, then every row-wise and transposing operand
//     read, and check that each returns the element its MFMA operand needs;
//   - the tiled copy the register-fed passes stream (mfma_layout.h tile_row /
//     tile_col): the 16 bytes a lane loads at k-step kk are the A operand of
//     the 16x16x32 logit product (row lane % 16, columns 32 kk + 8 (lane / 16)
//     .. + 7 of the wave's slice);
//   - the wide tiling: each wave writes those operand registers into its LDS
//     slice and reads it back with the transposing read of its second product.
// Also counts LDS bank conflicts with the service model measured on gfx950:
// a 16-byte-per-lane access is served 8 lanes at a time over 32 banks of 4
// bytes, the 8-byte transposing read 32 lanes at a time over 64 banks.
// Transposing read semantics (ds_read_b64_tr_b16, per 16-lane group): lane i
// receives, as element y, the 16-bit value (i % 4) of the 8 bytes addressed by
// lane 4 y + i / 4 of its group.
#include <algorithm>
#include <cstdio>
#include <map>
#include <set>
#include <utility>
#include <vector>

#include "mfma_layout.h"
#include "mfma_layout_wide.h"

using namespace solo::layout;

// Extra service passes caused by bank conflicts: lanes are served in groups
// of `pass` lanes; within a group, a bank holding k distinct dwords costs k - 1.
static int conflicts(const int* addr, int width, int pass, int nbanks) {
    int extra = 0;
    for (int p = 0; p < 64; p += pass) {
        std::map<int, std::set<int>> banks;
        for (int l = p; l < p + pass; ++l)
            for (int wd = 0; wd < width / 4; ++wd) banks[(addr[l] / 4 + wd) % nbanks].insert(addr[l] / 4 + wd);
        int worst = 1;
        for (auto& b : banks) worst = std::max(worst, (int)b.second.size());
        extra += worst - 1;
    }
    return extra;
}

// The operand a lane of wave w (DS columns per wave) holds after loading
// k-step kk of a chunk from the tiled copy: (row, column) of element e.
template <int DS>
static std::pair<int, int> loaded(int w, int kk, int lane, int e) {
    const int o = w * (DS / 32) * 64 + kk * 64 + lane;  // granule index inside the chunk
    return {tile_row(o), tile_col(o) + e};
}

// The tiled copy hands every lane of every wave its logit-product operand.
template <int DS, int NWAVES>
int check_tiled() {
    int errors = 0;
    for (int w = 0; w < NWAVES; ++w)
        for (int kk = 0; kk < DS / 32; ++kk)
            for (int l = 0; l < 64; ++l)
                for (int e = 0; e < 8; ++e)
                    if (loaded<DS>(w, kk, l, e) != std::pair<int, int>{l & 15, w * DS + 32 * kk + 8 * (l >> 4) + e})
                        ++errors;
    return errors;
}

// NWAVES waves of DS columns each cover the row width d = NWAVES DS.
template <int DS, int NWAVES>
int check(int& conflicts_row, int& conflicts_tr) {
    using G = Geo<DS>;
    const int d = DS * NWAVES;
    int errors = 0;
    conflicts_row = conflicts_tr = 0;
    for (int w = 0; w < NWAVES; ++w) {
        const int js = w * DS;
        // LDS byte -> (row, column) of the bf16 element stored there
        std::map<int, std::pair<int, int>> lds;
        for (int q = 0; q < G::NI; ++q) {
            for (int lane = 0; lane < 64; ++lane) {
                const int elem = stream_row0<DS>(q) * d + stream_voff<DS>(stream_vidx<DS>(q), d, js, lane) / 2;
                const int row = elem / d, col = elem % d;
                const int addr = stream_lds_off<DS>(q) + 16 * lane;
                if (addr < 0 || addr + 16 > G::SLICE) ++errors;
                for (int e = 0; e < 8; ++e) {
                    if (lds.count(addr + 2 * e)) ++errors;  // two granules written to one place
                    lds[addr + 2 * e] = {row, col + e};
                }
            }
        }
        if ((int)lds.size() != 16 * DS) ++errors;  // every element of the 16 x DS slice exactly once
        // row-wise reads: lane -> row lane % 16, columns js + 32 kk + 8 (lane / 16) + e
        for (int kk = 0; kk < DS / 32; ++kk) {
            int addr[64];
            for (int l = 0; l < 64; ++l) {
                const int base = rowread_off<DS>(l) + 64 * kk;
                addr[l] = base;
                for (int e = 0; e < 8; ++e) {
                    auto it = lds.find(base + 2 * e);
                    std::pair<int, int> want{l & 15, js + 32 * kk + 8 * (l >> 4) + e};
                    if (it == lds.end() || it->second != want) ++errors;
                }
            }
            conflicts_row += conflicts(addr, 16, 8, 32);
        }
        // transposing reads of block b: lane -> m = column js + 32 b + lane % 32,
        // k = rows 8 (lane / 32) + 4 half + y
        for (int b = 0; b < DS / 32; ++b) {
            for (int half = 0; half < 2; ++half) {
                int addr[64];
                for (int l = 0; l < 64; ++l) addr[l] = trread_off<DS>(l, half) + 64 * b;
                conflicts_tr += conflicts(addr, 8, 32, 64);
                for (int l = 0; l < 64; ++l) {
                    const int grp = l / 16, i = l % 16;
                    for (int y = 0; y < 4; ++y) {
                        const int src = grp * 16 + 4 * y + i / 4;
                        auto it = lds.find(addr[src] + 2 * (i % 4));
                        std::pair<int, int> want{8 * (l >> 5) + 4 * half + y, js + 32 * b + (l % 32)};
                        if (it == lds.end() || it->second != want) ++errors;
                    }
                }
            }
        }
    }
    return errors;
}

template <int DS, int NWAVES = NW>
int report() {
    int cr = 0, ct = 0;
    const int e = check<DS, NWAVES>(cr, ct);
    const int et = check_tiled<DS, NWAVES>();
    std::printf("DS=%d waves=%d padded=%d slice=%d errors=%d row_conflicts=%d tr_conflicts=%d tiled_errors=%d\n", DS,
                NWAVES, (int)Geo<DS>::PADDED, Geo<DS>::SLICE, e, cr, ct, et);
    return e + et;
}


// The wide layout (mfma_layout_wide.h): the operand registers of k-step kk
// written at the row-wise read offset of the slice, and the transposing reads
// of the 16x16x16 second product.
template <int DS>
int check_wide(int& conflicts_wr, int& conflicts_tr) {
    namespace W = solo::layoutw;
    using G = W::Geo<DS>;
    int errors = 0;
    conflicts_wr = conflicts_tr = 0;
    for (int w = 0; w < W::NW; ++w) {
        const int js = w * DS;
        std::map<int, std::pair<int, int>> lds;  // LDS byte -> (row, column within the slice)
        for (int kk = 0; kk < DS / 32; ++kk) {
            int addr[64];
            for (int l = 0; l < 64; ++l) {
                const int a = W::rowread_off<DS>(l, kk);
                addr[l] = a;
                if (a < 0 || a + 16 > G::SLICE) ++errors;
                for (int e = 0; e < 8; ++e) {
                    const std::pair<int, int> v = loaded<DS>(w, kk, l, e);
                    if (v != std::pair<int, int>{l & 15, js + 32 * kk + 8 * (l >> 4) + e}) ++errors;
                    if (lds.count(a + 2 * e)) ++errors;
                    lds[a + 2 * e] = {v.first, v.second - js};
                }
            }
            conflicts_wr += conflicts(addr, 16, 8, 32);
        }
        if ((int)lds.size() != 16 * DS) ++errors;
        for (int b = 0; b < DS / 16; ++b) {
            int addr[64];
            for (int l = 0; l < 64; ++l) addr[l] = W::trread_off<DS>(l, b);
            conflicts_tr += conflicts(addr, 8, 32, 64);
            for (int l = 0; l < 64; ++l) {
                const int grp = l / 16, i = l % 16;
                for (int e = 0; e < 4; ++e) {
                    const int src = grp * 16 + 4 * e + i / 4;
                    auto it = lds.find(addr[src] + 2 * (i % 4));
                    std::pair<int, int> want{4 * grp + e, 16 * b + i};  // A[m = column][k = row] of the 16x16x16 product
                    if (it == lds.end() || it->second != want) ++errors;
                }
            }
        }
    }
    return errors;
}

template <int DS>
int report_wide() {
    int cw = 0, ct = 0;
    const int e = check_wide<DS>(cw, ct);
    std::printf("WIDE DS=%d slice=%d errors=%d write_conflicts=%d tr_conflicts=%d\n", DS,
                solo::layoutw::Geo<DS>::SLICE, e, cw, ct);
    return e;
}

int main() {
    int e = 0;
    e += report<32>();
    e += report<64>();
    e += report<96>();
    e += report<128>();
    e += report<160>();
    e += report<192>();
    e += report<224>();
    e += report<256>();
    // the wide layout: 8 waves of d / 8 columns; 320 is the shipped width (d = 2560)
    e += report_wide<320>();
    e += report_wide<384>();
    return e == 0 ? 0 : 1;
}
