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
constexpr int kWaves = 8;          // waves per workgroup of the forward kernels
constexpr int kThreads = kWaves * 64;
constexpr int kAccPad = 17;        // fp32 stride of one accumulator row in LDS
constexpr int kMaxSkinnyM = 64;    // 4 m-tiles of 16
constexpr int kMaxGemvM = 8;
constexpr size_t kLdsMax = 160 * 1024 - 512;   // dynamic LDS per workgroup (static use is tiny)

enum Path { kAuto = 0, kGemv = 1, kSkinny = 2, kTiled = 3 };

// Arguments of one forward launch.  The K range [0, Kb) of groups is cut into
// S chunks and the Nt column tiles into Gn ranges; workgroup b handles chunk
// b / Gn and column range b % Gn.
struct FwdArgs {
    const uint4 *codes;     // device layout, Nt * Kb blocks of 1 KiB
    const void *sz;         // per (tile, group, column): u32 s | z << 16, or u16 s (symmetric)
    const uint16_t *x;      // [M][K] bf16
    uint16_t *y;            // [M][N] bf16
    float *ws;              // [S][M][N] fp32 partial sums (S > 1)
    uint32_t *counters;     // [Gn] arrival counters (S > 1), zero between launches
    int M, K, N, Kb, Nt, S, Gn;
};

// LDS bytes a forward workgroup needs (x chunk of Kc groups + accumulators of
// Tn column tiles).  `rows` = M for GEMV, 16 * m-tiles for SKINNY.
inline size_t lds_bytes(int path, int rows, int Kc, int Tn) {
    size_t xbytes = (path == kGemv) ? (size_t)rows * Kc * 256 : (size_t)Kc * rows * 256;
    return xbytes + (size_t)Tn * rows * kAccPad * 4;
}

// Host launchers (kernels.hip).  Each returns the launch status.
hipError_t launch_repack(const uint32_t *canon, const uint16_t *scales, const uint16_t *zeros,
                         uint4 *codes, void *sz, int K, int N, bool symmetric, hipStream_t st);
hipError_t launch_forward(int path, int mrows, bool symmetric, int grid, size_t lds,
                          const FwdArgs &a, hipStream_t st);
hipError_t launch_unpack(const uint4 *codes, uint8_t *q, int K, int N, hipStream_t st);
hipError_t launch_dequant(int routine, const uint4 *codes, const void *sz, bool symmetric,
                          uint16_t *w, int K, int N, hipStream_t st);
hipError_t prepare_kernels();     // per-process attribute setup (LDS limits)
const char *kernel_name(int path, int mrows, bool symmetric);

}  // namespace qlin
