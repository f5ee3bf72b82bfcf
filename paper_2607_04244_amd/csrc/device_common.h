// Device-side building blocks shared by the forward kernels (kernels.hip,
// tiled.hip): vector types, the block layout, the nibble extraction and the
// two exact dequantization routes.  Header-only, inline.
#pragma once

#include "qlin_internal.h"

namespace qlin {

typedef __attribute__((address_space(3))) void lds_void_t;   // LDS, for direct-to-LDS loads
typedef __attribute__((address_space(1))) void glb_void_t;   // global memory

typedef short v4s __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ layout

// Column (within the tile) and k (within the group) of nibble p of word j of lane l.
__host__ __device__ inline void block_coord(int l, int j, int p, int &n16, int &k128) {
    const int r = 2 * (p & 1) + (p >> 2);
    const int h = (p >> 1) & 1;
    n16 = 4 * ((l >> 2) & 3) + r;
    k128 = 32 * j + 8 * (l >> 4) + 4 * h + (l & 3);
}

// Buffer-resource constants.  Cross-workgroup partial sums travel between
// workgroups that may sit on different XCDs, whose L2 caches are not coherent
// with each other for ordinary accesses: they are written and read with
// agent-scope (sc1) buffer accesses, which the hardware performs at the
// device coherence point.
constexpr int kSc1 = 16;                 // cache-policy operand of the buffer builtins: sc1 (agent scope)
constexpr int kRsrcFlags = 0x00020000;   // buffer descriptor word 3: 32-bit raw data

// ------------------------------------------------------------------ small helpers

__device__ inline uint32_t cvt_pk_bf16(float lo, float hi) {
    v2f f = {lo, hi};
    v2bf b = __builtin_convertvector(f, v2bf);   // round to nearest even
    return __builtin_bit_cast(uint32_t, b);
}

__device__ inline uint16_t cvt_bf16(float v) {
    __bf16 b = (__bf16)v;
    return __builtin_bit_cast(uint16_t, b);
}

__device__ inline float bf16_lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// The four "128 + q" bf16 pairs of one packed word: pair i holds nibbles i
// (low half) and i + 4 (high half).  Each pair is one v_and_or_b32; the two
// constants live in registers (gfx9 VOP3 takes no literal), loaded once per
// kernel by ExtractConsts.
struct ExtractConsts {
    uint32_t mask, magic;
    __device__ inline ExtractConsts() {
        // opaque to the optimizer, so the values stay in registers
        mask = __builtin_amdgcn_readfirstlane(0x000F000Fu);
        magic = 0x43004300u;                        // bf16 128.0 in both halves
        asm volatile("" : "+v"(magic));
    }
};
struct Pairs { uint32_t a0, a1, a2, a3; };
__device__ inline Pairs extract_pairs(uint32_t P, const ExtractConsts &k) {
    Pairs o;
    o.a0 = (P & k.mask) | k.magic;
    o.a1 = ((P >> 4) & k.mask) | k.magic;
    o.a2 = ((P >> 8) & k.mask) | k.magic;
    o.a3 = ((P >> 12) & k.mask) | k.magic;
    return o;
}

// One lane's 16 bytes of a weight block.
__device__ inline uint4 load_block(const uint4 *codes, size_t idx) { return codes[idx]; }

// Cache policy of the decode kernels' weight loads: non-temporal.  A forward
// reads every weight once, so streaming them with this hint keeps them from
// displacing x, y and the partial sums in L2 and the last-level cache (the
// tiled kernel keeps ordinary loads: the row blocks of a column block reuse
// its weights from L2).
constexpr int kWeightPolicy = 2;   // cache-policy operand of the buffer builtins: nt
__device__ inline uint4 load_block_nt(const uint4 *codes, size_t idx) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load((const v4u *)codes + idx));
}

// Per (column, group) dequantization word: bf16 s in the low half and the
// bf16 offset zc = -(128 + z) in the high half (exact: an integer of 8
// significant bits), so that (128 + q) * s + zc * s = (q - z) * s.
// Symmetric handles store only s (z = 8, zc = -136 = bf16 0xC308).
constexpr uint32_t kZcSymmetric = 0xC308u;
template <bool SYM>
__device__ inline uint32_t load_sz(const void *sz, size_t idx) {
    if constexpr (SYM) {
        return (uint32_t)((const uint16_t *)sz)[idx] | (kZcSymmetric << 16);
    } else {
        return ((const uint32_t *)sz)[idx];
    }
}

template <bool SYM>
__device__ inline uint32_t load_sz_nt(const void *sz, size_t idx) {   // non-temporal, as load_block_nt
    if constexpr (SYM) {
        return (uint32_t)__builtin_nontemporal_load((const uint16_t *)sz + idx) | (kZcSymmetric << 16);
    } else {
        return __builtin_nontemporal_load((const uint32_t *)sz + idx);
    }
}

__device__ inline float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(v2bf, a), __builtin_bit_cast(v2bf, b), c, false);
}

// c = s * zc of a dequantization word, exactly (one bf16 product, plus 0)
__device__ inline float sz_offset(uint32_t sz) { return dot2(sz, sz >> 16, 0.0f); }

// --- matrix-core dequantization ------------------------------------------

struct MfmaDeq { v4s bdiag; v4f c4; };

// Byte selectors (v_perm_b32) that place the bf16 s of a dequantization
// word into element l & 3 of lane l's B operand (two dwords, four bf16) and
// zero the other three elements.  Constant per lane; built once per kernel.
struct DiagSel {
    uint32_t s0, s1;
    __device__ inline explicit DiagSel(int lane) {
        constexpr uint32_t kLo = 0x0C0C0100u, kHi = 0x01000C0Cu, kZero = 0x0C0C0C0Cu;
        const int r = lane & 3;
        s0 = r == 0 ? kLo : r == 1 ? kHi : kZero;
        s1 = r == 2 ? kLo : r == 3 ? kHi : kZero;
    }
};

// Per-group constants of lane l for column n = 16 t + (l & 15):
// B = diag(s) in the 4x4 block layout (this lane supplies B[r][l & 3],
// non-zero only for r = l & 3) and C = zc * s = -(128 + z) * s in all four rows.
__device__ inline MfmaDeq mfma_setup(uint32_t sz, const DiagSel &sel) {
    const float c = sz_offset(sz);
    MfmaDeq d;
    d.bdiag = __builtin_bit_cast(v4s, v2u{__builtin_amdgcn_perm(sz, sz, sel.s0), __builtin_amdgcn_perm(sz, sz, sel.s1)});
    d.c4 = v4f{c, c, c, c};
    return d;
}

// Dequantize one packed word into the 8 bf16 A-operand values of
// v_mfma_f32_16x16x32_bf16 (row n = l & 15): element e holds
// w[n][32j + 8(l >> 4) + e].
__device__ inline v8bf mfma_dequant(uint32_t P, const MfmaDeq &d, const ExtractConsts &k) {
    const Pairs a = extract_pairs(P, k);
    const v4s A0 = __builtin_bit_cast(v4s, v2u{a.a0, a.a1});
    const v4s A1 = __builtin_bit_cast(v4s, v2u{a.a2, a.a3});
    const v4f d0 = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(A0, d.bdiag, d.c4, 0, 0, 0);
    const v4f d1 = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(A1, d.bdiag, d.c4, 0, 0, 0);
    const v4u w = {cvt_pk_bf16(d0[0], d0[1]), cvt_pk_bf16(d0[2], d0[3]),
                   cvt_pk_bf16(d1[0], d1[1]), cvt_pk_bf16(d1[2], d1[3])};
    return __builtin_bit_cast(v8bf, w);
}

// --- vector-ALU dequantization -------------------------------------------

// Constants for the four columns n = 16 t + 4 * ((l >> 2) & 3) + r of lane l.
struct ValuDeq { uint32_t sl[4], sh[4]; float c[4]; };

__device__ inline ValuDeq valu_setup(const uint32_t sz[4]) {
    ValuDeq d;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        d.c[r] = sz_offset(sz[r]);   // -(128 + z) * s
        d.sl[r] = sz[r] & 0xFFFFu;   // bf16 pair (s, 0)
        d.sh[r] = sz[r] << 16;       // bf16 pair (0, s)
    }
    return d;
}

// Dequantize one packed word: pr[r] = bf16 pair (w[n_r][k0], w[n_r][k0 + 4]) with
// k0 = 32j + 8(l >> 4) + (l & 3).
__device__ inline void valu_dequant(uint32_t P, const ValuDeq &d, const ExtractConsts &k, uint32_t pr[4]) {
    const Pairs a = extract_pairs(P, k);
    const float w00 = dot2(a.a0, d.sl[0], d.c[0]), w01 = dot2(a.a0, d.sh[1], d.c[1]);
    const float w02 = dot2(a.a1, d.sl[2], d.c[2]), w03 = dot2(a.a1, d.sh[3], d.c[3]);
    const float w10 = dot2(a.a2, d.sl[0], d.c[0]), w11 = dot2(a.a2, d.sh[1], d.c[1]);
    const float w12 = dot2(a.a3, d.sl[2], d.c[2]), w13 = dot2(a.a3, d.sh[3], d.c[3]);
    pr[0] = cvt_pk_bf16(w00, w10);
    pr[1] = cvt_pk_bf16(w01, w11);
    pr[2] = cvt_pk_bf16(w02, w12);
    pr[3] = cvt_pk_bf16(w03, w13);
}

// ------------------------------------------------------------------ LDS staging

// One direct-to-LDS 16-byte load per lane: lane l's 16 bytes from src land
// at lds_dst + 16 l (lds_dst uniform across the wave).  Issued as inline
// assembly so that the compiler does not track it: its wait-count pass
// handles direct-to-LDS writes coarsely and would drain every outstanding
// load before each later LDS read.  The caller waits for it explicitly
// (s_waitcnt vmcnt) before the barrier that publishes the data; loads the
// compiler does track and issues later are younger, so its own waits stay
// sufficient.  These statements set m0 themselves and list it as clobbered;
// the compiler warns that it may not preserve a reserved register across
// them, which matters only if it kept a value of its own in m0: the
// generated code of every kernel here has no other m0 access.
__device__ inline void load_lds_x16(const void *src, const uint4 *lds_dst) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" :: "s"(m0), "v"(src) : "memory", "m0");
}

// The same with the non-temporal hint, for data a call reads once.
__device__ inline void load_lds_x16_nt(const void *src, const uint4 *lds_dst) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off nt" :: "s"(m0), "v"(src) : "memory", "m0");
}

// The same with 4 bytes per lane: lane l's dword lands at lds_dst + 4 l.
__device__ inline void load_lds_x4(const void *src, const void *lds_dst) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst);
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" :: "s"(m0), "v"(src) : "memory", "m0");
}

// LDS byte address of p (wave-uniform), as a scalar.
__device__ inline uint32_t lds_addr(const void *p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p);
}

// Direct-to-LDS buffer loads: lane l's 16 (4) bytes at byte offset
// voff + soff of the resource land at LDS byte address lds + 16 l (4 l).
// Inline assembly for the same reason as load_lds_x16; lds and soff are
// scalars, so a load whose per-lane offset is fixed costs no vector work.
__device__ inline void load_lds_buf16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
__device__ inline void load_lds_buf4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}

// Barrier for LDS hand-off only.  __syncthreads() also waits for every
// outstanding global load, which would drain the weight prefetch.
__device__ inline void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace qlin
