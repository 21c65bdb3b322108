// Device helpers of the matrix-core passes (k_mfma.hip, k_mfma_wide.hip):
// operand types, MFMA wrappers, the direct-to-LDS chunk stream, row
// reductions over lane groups and the waits that go with the untracked stream.
#pragma once

#include "mfma_layout.h"
#include "solo_internal.h"

namespace solo {
namespace mfma {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

// Logits are handled in base 2 (z2 = z log2 e), so each probability costs one
// v_exp_f32.  The running max is re-based only when a logit exceeds it by more
// than kLazyThresh2 (probabilities then stay below 2^kLazyThresh2), which after
// the first chunk almost never happens: the common path needs no row maximum.
constexpr float kLog2e = 1.44269504088896341f;
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLazyThresh2 = 11.0f;

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float bf16_bits_to_f32(unsigned short u) {
    return __uint_as_float(((unsigned)u) << 16);
}

// Direct buffer -> LDS load of 16 bytes per lane; lane l's bytes land at
// lds_base + 16 l.  Issued as inline asm so that the compiler does not track
// it: the only reader of a chunk is the next step, which starts after an
// explicit vmcnt(0) wait (wait_vm), and without tracking the compiler adds no
// conservative waits before unrelated LDS accesses.  M0 (the LDS base of the
// transfer) is a register the compiler reserves, so it is saved and restored;
// one wait state separates an M0 write from the LDS-DMA that reads it.
__device__ __forceinline__ void buffer_load_lds16(i32x4 rsrc, unsigned lds_base, int voffset) {
    unsigned saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voffset), "s"(rsrc)
        : "memory");
}

// Same for 4 bytes per lane: lane l's dword lands at lds_base + 4 l.
__device__ __forceinline__ void buffer_load_lds4(i32x4 rsrc, unsigned lds_base, int voffset) {
    unsigned saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dword %2, %3, 0 offen lds\n\t"
        "s_nop 0\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voffset), "s"(rsrc)
        : "memory");
}

// The end of one row's online softmax, in base 2.  The running sum sx holds
// every column but the target's: sx = sum_{v != y} 2^(z_v - m), with m the
// (lazily re-based) running maximum and zy the target's logit.  Adding the
// target's term 2^(zy - m) only here gives p_y - 1 = -sx / s and the row loss
// without cancellation even where the target holds nearly all of the
// probability: loss = log(1 + sx / e_y) then, (m - zy) ln 2 + ln s otherwise.
// An invalid target (tok false) has no target term: NaN loss, no one-hot term.
struct RowEnd {
    float lse2;   // log-sum-exp, base 2
    float loss;   // row loss, nats
    float py1;    // p_y - 1 (0 without a valid target)
    float inv_s;  // 1 / sum_v 2^(z_v - m)
};
__device__ __forceinline__ RowEnd finish_row(float m, float sx, float zy, bool tok) {
    const float ey = tok ? __builtin_amdgcn_exp2f(zy - m) : 0.f;
    const float s = sx + ey;
    RowEnd o;
    o.lse2 = m + __log2f(s);
    o.inv_s = 1.f / s;
    o.py1 = tok ? -sx * o.inv_s : 0.f;
    o.loss = !tok ? __int_as_float(0x7fc00000) : (ey > sx ? log1pf(sx / ey) : ((m - zy) + __log2f(s)) * kLn2);
    return o;
}

// All-lane reductions over each 16-lane row of the wave (DPP: quad
// permutations, then rotations by 4 and 8 inside the row).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp_f<0xB1>(x));   // quad_perm [1,0,3,2]
    x = fmaxf(x, dpp_f<0x4E>(x));   // quad_perm [2,3,0,1]
    x = fmaxf(x, dpp_f<0x124>(x));  // row_ror:4
    x = fmaxf(x, dpp_f<0x128>(x));  // row_ror:8
    return x;
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x124>(x);
    x += dpp_f<0x128>(x);
    return x;
}

// The same over each group of 8 lanes (quad permutations, then the mirror
// inside each half row), and the choice between the two by group size.
__device__ __forceinline__ float row8_max(float x) {
    x = fmaxf(x, dpp_f<0xB1>(x));   // quad_perm [1,0,3,2]
    x = fmaxf(x, dpp_f<0x4E>(x));   // quad_perm [2,3,0,1]
    x = fmaxf(x, dpp_f<0x141>(x));  // row_half_mirror
    return x;
}
__device__ __forceinline__ float row8_sum(float x) {
    x += dpp_f<0xB1>(x);
    x += dpp_f<0x4E>(x);
    x += dpp_f<0x141>(x);
    return x;
}
template <int N>
__device__ __forceinline__ float group_max(float x) {
    static_assert(N == 8 || N == 16, "lane groups of 8 or 16");
    return N == 16 ? row16_max(x) : row8_max(x);
}
template <int N>
__device__ __forceinline__ float group_sum(float x) {
    static_assert(N == 8 || N == 16, "lane groups of 8 or 16");
    return N == 16 ? row16_sum(x) : row8_sum(x);
}

// The lane index, produced by a volatile instruction: an address computed
// from it cannot be hoisted out of a loop, so it is recomputed (a few cheap
// instructions) where it is used instead of holding a register for the whole
// loop (the widest passes have none to spare).
__device__ __forceinline__ int lane_now() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
}

__device__ __forceinline__ unsigned lds_addr(LDS_AS char* p) {
    return __builtin_amdgcn_readfirstlane((unsigned)(unsigned long long)p);
}

// Buffer resource over [base, base + bytes): loads at or beyond `bytes`
// return zeros, which pads the ragged last chunk.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, unsigned bytes) {
    const unsigned long long a = (unsigned long long)base;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(unsigned)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(unsigned)(a >> 32));
    r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
    r[3] = 0x00020000;
    return r;
}

// The direct-to-LDS stream of one chunk (layout in mfma_layout.h).
template <int DS>
struct ChunkStream {
    using G = layout::Geo<DS>;
    int voff[G::NV];

    __device__ __forceinline__ void init(int d, int js, int lane) {
#pragma unroll
        for (int v = 0; v < G::NV; ++v) voff[v] = layout::stream_voff<DS>(v, d, js, lane);
    }

    // buffer resource of the chunk starting at row y0; rows at or beyond nY
    // read as zeros.  The range covers this chunk only: one over all remaining
    // rows would pass 2^32 bytes (and wrap) for long matrices.
    __device__ __forceinline__ static i32x4 rsrc(const bf16* __restrict__ Y, int nY, int d, int y0) {
        const int rows = nY - y0 < layout::YC ? nY - y0 : layout::YC;
        const unsigned rem = rows > 0 ? (unsigned)rows * (unsigned)d * 2u : 0u;
        return make_rsrc(Y + (long long)(rows > 0 ? y0 : 0) * d, rem);
    }

    // instructions [Q0, Q1) of the stream of one chunk into `slice`
    template <int Q0, int Q1>
    __device__ __forceinline__ void issue_range(i32x4 rs, int d, unsigned slice) const {
#pragma unroll
        for (int q = Q0; q < Q1; ++q) {
            const int voffset = voff[layout::stream_vidx<DS>(q)] + layout::stream_row0<DS>(q) * d * 2;
            buffer_load_lds16(rs, slice + layout::stream_lds_off<DS>(q), voffset);
        }
    }

    // instruction q alone (q a constant after unrolling)
    __device__ __forceinline__ void issue_one(i32x4 rs, int d, unsigned slice, int q) const {
        const int voffset = voff[layout::stream_vidx<DS>(q)] + layout::stream_row0<DS>(q) * d * 2;
        buffer_load_lds16(rs, slice + layout::stream_lds_off<DS>(q), voffset);
    }

    // stream rows y0 .. y0 + 15 (this wave's DS columns) of Y into `slice`
    __device__ __forceinline__ void issue(const bf16* __restrict__ Y, int nY, int d, int y0, unsigned slice) const {
        issue_range<0, G::NI>(rsrc(Y, nY, d, y0), d, slice);
    }
};

// Barrier for LDS traffic only: unlike __syncthreads it does not drain the
// in-flight chunk prefetch.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// vmcnt(0) (expcnt and lgkmcnt not waited for: gfx9 encoding 0x0F70) through
// the builtin, so that the compiler's own wait tracking sees it too, followed
// by a compiler barrier that keeps LDS reads of the new chunk below it.
__device__ __forceinline__ void wait_vm() {
    __builtin_amdgcn_s_waitcnt(0x0F70);
    asm volatile("" ::: "memory");
}


}  // namespace mfma
}  // namespace solo
