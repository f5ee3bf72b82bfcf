// Internal interface between the C-ABI host code (qlin.cpp) and the HIP
// kernels (kernels.hip).  Not installed; the public ABI is include/qlin.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace qlin {

constexpr int kGroup = 128;        // K elements per quantization group
constexpr int kTileN = 16;         // output columns per weight tile
constexpr int kBlockU32 = 256;     // packed words per (16 n x 128 k) block = 1 KiB
#ifndef QLIN_WAVES
#define QLIN_WAVES 8
#endif
#ifndef QLIN_DEPTH
#define QLIN_DEPTH 4
#endif
constexpr int kWaves = QLIN_WAVES; // waves per workgroup of the forward kernels
constexpr int kDepth = QLIN_DEPTH; // 1 KiB weight blocks in flight per wave
constexpr int kThreads = kWaves * 64;
constexpr int kMaxSkinnyM = 64;    // 4 m-tiles of 16
constexpr int kMaxGemvM = 4;
constexpr int kTnMax = 8;          // column tiles per workgroup, register-resident kernels
constexpr int kTnMaxGemv = 4;      // the same for the vector-ALU GEMV kernel
constexpr size_t kLdsMax = 160 * 1024 - 512;   // dynamic LDS per workgroup (static use is tiny)
constexpr int kXChunksMax = 8192;  // 16-byte x chunks one workgroup stages (128 KiB)

enum Path { kAuto = 0, kGemv = 1, kSkinny = 2, kTiled = 3 };

// Kernel families behind the paths (host planning, launch selection).
enum Kern {
    kKernGemv = 0,     // k_gemv4: M <= 4, group-major, x in registers
    kKernMfma16 = 1,   // k_mfma16: M <= 16, group-major, x in registers
    kKernStaged = 2    // k_skinny<MT>: 16 < M <= 64, x chunk staged in LDS
};

// Arguments of one forward launch.  The K range [0, Kb) of groups is cut into
// S chunks and the Nt column tiles into Gn ranges; workgroup b handles chunk
// b / Gn and column range b % Gn.  Range j holds Nq (+1 for j < Nr) tiles
// and chunk c holds Kq (+1 for c < Kr) groups, so the kernels need no
// division to find their work.
struct FwdArgs {
    const uint4 *codes;     // device layout, Nt * Kb blocks of 1 KiB
    const void *sz;         // per (tile, group, column): u32 s | z << 16, or u16 s (symmetric)
    const uint16_t *x;      // [M][K] bf16
    uint16_t *y;            // [M][N] bf16
    float *ws;              // [S][M][N] fp32 partial sums (S > 1)
    uint32_t *counters;     // [Gn] arrival counters (S > 1), zero between launches
    int M, K, N, Kb, Nt, S, Gn;
    int Nq, Nr, Kq, Kr;
};
static_assert((kWaves & (kWaves - 1)) == 0, "waves per workgroup must be a power of two");

// x chunks of a K chunk of Kc groups with `rows` staged rows
inline int x_chunks(int rows, int Kc) { return rows * Kc * 16; }

// LDS bytes of the register-resident kernels: one slot of rows x 16 fp32
// per (wave, tile).
inline size_t lds_bytes_regs(int rows) { return (size_t)kWaves * kTnMax * rows * 16 * 4; }

// LDS bytes a forward workgroup needs: the x chunk of Kc groups plus one
// partial-sum slot (rows x 16 fp32) per (wave, column tile) pair a wave
// touches; slot = wave + tile is unique, so kWaves + Tn - 1 slots suffice.
// `rows` = M for GEMV, 16 * m-tiles for SKINNY.
inline size_t lds_bytes(int path, int rows, int Kc, int Tn) {
    (void)path;
    return (size_t)Kc * rows * 256 + (size_t)(kWaves + Tn) * rows * 16 * 4;
}

// Host launchers (kernels.hip).  Each returns the launch status.
hipError_t launch_repack(const uint32_t *canon, const uint16_t *scales, const uint16_t *zeros,
                         uint4 *codes, void *sz, int K, int N, bool symmetric, hipStream_t st);
hipError_t launch_forward(int kern, int mrows, bool symmetric, int grid, size_t lds,
                          const FwdArgs &a, hipStream_t st);
hipError_t launch_unpack(const uint4 *codes, uint8_t *q, int K, int N, hipStream_t st);
hipError_t launch_dequant(int routine, const uint4 *codes, const void *sz, bool symmetric,
                          uint16_t *w, int K, int N, hipStream_t st);
hipError_t prepare_kernels();     // per-process attribute setup (LDS limits)
hipError_t launch_stream_read(const void *buf, size_t bytes, int grid, uint32_t *sink, hipStream_t st);
const char *kernel_name(int kern, int mrows, bool symmetric);

}  // namespace qlin
