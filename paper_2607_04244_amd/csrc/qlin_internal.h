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
#define QLIN_DEPTH 3
#endif
constexpr int kWaves = QLIN_WAVES; // waves per workgroup of the forward kernels
constexpr int kDepth = QLIN_DEPTH; // 1 KiB weight blocks in flight per wave
constexpr int kThreads = kWaves * 64;
constexpr int kMaxSkinnyM = 64;    // 4 m-tiles of 16
constexpr int kMaxGemvM = 4;
constexpr int kTnMax = 8;          // column tiles per workgroup, register-resident kernels
constexpr int kTnMaxGemv = 4;      // the same for the vector-ALU GEMV kernel
constexpr size_t kLdsMax = 160 * 1024 - 512;   // dynamic LDS per workgroup (static use is tiny)

enum Path { kAuto = 0, kGemv = 1, kSkinny = 2, kTiled = 3, kRegs = 4 };

// Kernel families behind the paths (host planning, launch selection).
enum Kern {
    kKernGemv = 0,     // k_gemv4: M <= 4, group-major walk, x in registers (GEMV path)
    kKernMfma16 = 1,   // k_mfma16: M <= 16, group-major walk, x in registers (REGS path)
    kKernStaged = 2,   // k_skinny<MT>: M <= 64, tile-major walk, x chunk staged in LDS (SKINNY path)
    kKernTiled = 3     // k_tiled: any M, 128 x 256 output blocks, x and weights staged in LDS (TILED path)
};

// Arguments of one forward launch of the decode kernels, over one linear or
// over a group of up to kMaxMembers linears that share x (same K).  The K
// range [0, Kb) of groups is cut into S chunks and the column tiles of the
// members into Gn ranges in all; workgroup b handles chunk b / Gn and column
// range b % Gn.  Ranges [gn0, gn0 + its range count) belong to one member,
// whose Nt tiles they split as Nq (+1 for its first Nr ranges), so the
// kernels need no division to find their work.
constexpr int kMaxMembers = 8;
struct FwdMember {
    const uint4 *codes;     // device layout, Nt * Kb blocks of 1 KiB
    const void *sz;         // per (tile, group, column): u32 s | zc << 16 with zc = -(128 + z), or u16 s (symmetric)
    uint16_t *y;            // [M][N] bf16
    int N;                  // output columns
    int Nq, Nr;
};
struct FwdArgs {
    const uint16_t *x;      // [M][K] bf16, shared by all members
    float *ws;              // fp32 partial sums (S > 1): S * Gn regions of TnMax * M * 16
    uint32_t *counters;     // [Gn] arrival counters (S > 1), zero between launches
    int M, K, Kb, S, Gn;
    uint32_t inv_gn;        // ceil(2^32 / Gn) (0 for Gn = 1): chunk of workgroup b = umulhi(b, inv_gn)
    int Kq, Kr;
    int TnMax;              // tiles of the widest column range
    uint32_t ws_bytes;      // size of ws (bounds of its buffer descriptor)
    int nmem;               // members, 1 .. kMaxMembers
    int gn0[kMaxMembers];   // first column range of each member (Gn for absent members)
    FwdMember mem[kMaxMembers];
};
static_assert((kWaves & (kWaves - 1)) == 0, "waves per workgroup must be a power of two");

// TILED kernel (prefill-sized M): a workgroup of kTiledWaves x WS waves
// computes a (16 MSW) x (64 NT) block of y; wave w owns all 16 MSW rows of
// column tiles NW w .. NW w + NW - 1 (NW = NT / WS).  Block shapes (MSW, NT): 128 x 256
// (8, 4) and 64 x 128 (4, 2); the planner takes the large one when its
// blocks fill the last round of compute units well.
constexpr int kTiledWaves = 4;
constexpr int kTiledStages = 3;                            // LDS pipeline depth (groups)
struct TiledShape { int msw, nt; };
constexpr TiledShape kTiledShapes[] = {{8, 4}, {4, 2}, {6, 4}};
// Wave split of a shape: the 128 x 256 blocks run two waves per SIMD, each
// owning half of every column group's tiles.
constexpr int tiled_wsplit(TiledShape sh) { return sh.nt == 4 ? 2 : 1; }

// A tiled launch covers the column blocks of up to kMaxMembers linears that
// share x: member i owns column blocks [gb0[i], gb0[i + 1]) and its column
// tiles [0, Nt) are cut into blocks of 4 NT tiles from its first.
struct TiledMember {
    const uint4 *codes;
    const void *sz;
    uint16_t *y;            // [M][N] bf16
    int N, Nt;
};
struct TiledArgs {
    const uint16_t *x;      // [M][K] bf16
    int M, K, Kb;
    int Mt;                 // row blocks: ceil(M / (16 MSW))
    int Gn;                 // column blocks over all members
    int S;                  // K chunks; chunk c holds Kq (+1 for c < Kr) groups
    int Kq, Kr;
    float *ws;              // S > 1: fp32 partial blocks, Gn Mt S of 16 MSW x 64 NT
    uint32_t *counters;     // S > 1: [Gn Mt] arrival counters, zero between launches
    uint32_t ws_bytes;      // size of ws
    int nmem;
    int gb0[kMaxMembers];   // first column block of each member (Gn for absent members)
    TiledMember mem[kMaxMembers];
};

// Rows of x a SKINNY workgroup keeps in LDS for M rows (M <= 64): the next
// power of two >= M up to 16, else whole m-tiles of 16.
inline int staged_rows(int M) {
    if (M > 16) return 16 * ((M + 15) / 16);
    int r = 1;
    while (r < M) r <<= 1;
    return r;
}

// LDS bytes of the register-resident kernels with tn tile slots: one slot of
// rows x 16 fp32 per (wave, tile).
inline size_t lds_bytes_regs(int rows, int tn) { return (size_t)kWaves * tn * rows * 16 * 4; }

// LDS bytes of a SKINNY workgroup with M rows: the x chunk of Kc groups
// (staged_rows(M) rows of 16 Kc + 1 slots of 16 bytes, in whole 1 KiB
// direct-to-LDS loads) plus one
// partial-sum slot (16 m-columns per m-tile x 16 fp32) per (wave, column
// tile) pair.
inline size_t lds_bytes(int M, int Kc, int Tn) {
    const int mrows = 16 * ((M + 15) / 16);
    const size_t x = ((size_t)staged_rows(M) * (Kc * 16 + 1) * 16 + 1023) / 1024 * 1024;
    return x + (size_t)kWaves * Tn * mrows * 16 * 4;
}

// Host launchers (kernels.hip).  Each returns the launch status.
hipError_t launch_repack(const uint32_t *canon, const uint16_t *scales, const uint16_t *zeros,
                         uint4 *codes, void *sz, int K, int N, bool symmetric, hipStream_t st);
hipError_t launch_forward(int kern, int mrows, int tn, bool symmetric, int grid, size_t lds,
                          const FwdArgs &a, hipStream_t st);
hipError_t launch_unpack(const uint4 *codes, uint8_t *q, int K, int N, hipStream_t st);
hipError_t launch_dequant(int routine, const uint4 *codes, const void *sz, bool symmetric,
                          uint16_t *w, int K, int N, hipStream_t st);
hipError_t prepare_kernels();     // per-process attribute setup (LDS limits)
hipError_t launch_quantize(const uint16_t *w, const uint16_t *scales, const uint16_t *zeros, uint32_t *packed,
                           int K, int N, hipStream_t st);
hipError_t launch_tiled(bool symmetric, TiledShape shape, const TiledArgs &a, int grid, hipStream_t st);
hipError_t launch_stream_read(const void *buf, size_t bytes, int grid, uint32_t *sink, hipStream_t st);
const char *kernel_name(int kern, int mrows, int tn, bool symmetric);

// Static split-K scratch (kernels.hip) for callers that cannot allocate:
// kStaticScratchBytes per device, laid out as every workspace (counters,
// then partials).  static_scratch_setup looks up the array's device address
// on `device` (which must be current) once and clears its counters on st;
// static_scratch returns that address (NULL before the set-up).
constexpr size_t kStaticScratchBytes = (size_t)16 << 20;
constexpr size_t kScratchCounterBytes = (size_t)16 << 10;   // the counter region of every workspace
constexpr int kMaxDevices = 64;
hipError_t static_scratch_setup(int device, hipStream_t st);
void *static_scratch(int device);

// ---- error state shared by the C-ABI sources (defined in qlin.cpp)
int fail(int code, const char *fmt, ...);
int hip_fail(hipError_t e, const char *what);
void clear_err();
int last_status();

}  // namespace qlin
