// Internal interface between the C-ABI host code (spear_api.cpp) and the
// gfx950 kernels (spear_kernels.hip). Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace spear {

enum { DT_F16 = 0, DT_BF16 = 1 };
enum { GATE_ONE = 0, GATE_SIGMOID = 1, GATE_TANH = 2 };
// Epilogue variants of the 4-bit product kernels.
enum { EPI_NONE = 0,   // Y = X W^T
       EPI_READY = 1,  // Y = X W^T + v B^T, v already in the workspace
       EPI_FUSED = 2,  // same, v produced by EC workgroups of the same grid
       EPI_LOCAL = 3,  // same, [A; w_g] x computed by the GEMV waves themselves
       EPI_LOCAL_I8 = 4  // EPI_LOCAL with INT8 A and B (per-channel fp32 scales)
                       // over their K chunks (small rank), v from it per block
};
// How the EC projection's K-slices are combined.
enum { EC_LAST = 0,    // the last slice to arrive sums the partials, applies
                       // the gate and publishes v
       EC_GATHER = 1,  // fused only: every slice publishes its tagged partial
                       // sums; each consumer sums them and applies the gate
       EC_RAW = 2      // like EC_LAST, but publishes u = [A; w_g] x ungated
};

constexpr int kIterK = 128;      // K consumed per GEMV/EC iteration
constexpr int kTokTile = 16;     // tokens per MFMA token tile
constexpr int kEcTiles = 2;      // 16-row tiles of [A; w_g] per EC pass
constexpr int kGemmTM = 128;     // prefill tile: tokens
constexpr int kGemmTN = 128;     // prefill tile: output rows
constexpr int kGemmTK = 64;      // prefill tile: K per stage
constexpr int kGemmLdsRow = kGemmTK + 8;  // padded LDS row (halves)
constexpr int kVCopies = 8;      // copies of the published EC data (one per XCD)
constexpr int kLocalTiles = 2;   // EPI_LOCAL: B operands per iteration: A (r <= 16), w_g
constexpr size_t kLocalALds = 81920;  // EPI_LOCAL: LDS for the staged K-slice of A, w_g

// Workspace: a fixed counter block at the start, shared by every kind of call
// (the split-K and EC-slice counters return to zero after each call; the
// fused path's generation and ready counters advance by 2^32 per launch),
// then the region of the fused path's tagged words, which no other kind of
// call writes, then the call's data.
constexpr size_t kCounterBytes = 131072;
constexpr size_t kTagBytes = (size_t)1 << 20;         // fused path: tagged words
constexpr size_t kDataBase = kCounterBytes + kTagBytes;  // every call's data regions
constexpr size_t kCtrGen = 0;          // fused path: kGenClasses 64-bit launch
constexpr int kGenClasses = 64;        // counters, kGenStride apart
constexpr size_t kGenStride = 256;
constexpr size_t kCtrEc = 16384;       // EC-slice counters, one per token tile
constexpr int kMaxEcCounters = 4096;
constexpr size_t kCtrRows = 32768;     // split-K counters, one per row group / tile
constexpr size_t kCtrReady = 98304;    // fused path: kVCopies 64-bit ready
constexpr size_t kReadyStride = 4096;  // counters, 4 KB apart (memory channels)
constexpr int kMaxRowCounters = (int)((kCtrReady - kCtrRows) / 4);

// Launch generation of the fused path. Workgroup b belongs to counter class
// b % kGenClasses; every class counter advances by exactly 2^32 per launch:
// the class's first workgroup adds 2^32 - (members - 1) when it ends, every
// other member adds 1 (and workgroup 0 adds 2^32 to the classes no workgroup
// of a small grid belongs to). Any workgroup of launch L therefore reads a
// value in [L * 2^32, (L + 1) * 2^32) from its class counter when it starts,
// and the high word is the launch generation, with no workgroup waiting for
// another and no one address taking every workgroup's update.
__host__ __device__ inline uint64_t gen_increment(int block, int grid) {
  const int c = block % kGenClasses;
  const int members = (grid - c + kGenClasses - 1) / kGenClasses;
  return block < kGenClasses ? (1ull << 32) - (uint64_t)(members - 1) : 1ull;
}
// The ready counters advance by exactly 2^32 per launch too, summed over the
// publishers of the EC data (one per producer or per token tile), each adding
// its share (publisher_increment) once its data is complete: they read
// (g + 1) * 2^32 when every publisher of launch g is done.
__host__ __device__ inline uint64_t publisher_increment(int pub, int npub) {
  return pub == 0 ? (1ull << 32) - (uint64_t)(npub - 1) : 1ull;
}
// Tag of data published by the fused launch of generation g. The tagged
// words live in a workspace region that only fused launches write, so a word
// there is zero (never written) or was written by a fused launch of some
// generation g' <= g; its tag equals this launch's only if g' == g modulo
// 2^32 (g + 1 is never 0 before 2^32 - 1 launches have passed).
__host__ __device__ inline uint32_t ec_tag(uint32_t gen) { return gen + 1u; }

// EC projection / gate work. A producer workgroup owns one token tile (16
// tokens), one K-slice (ips iterations of 128) and one group of row tiles
// (tpg tiles of 16 rows of [A; w_g]).
struct EcParams {
  const uint16_t* x;      // [M][K]
  const uint16_t* A;      // [r][K] act dtype (null with INT8 A)
  const int8_t* A8;       // [r][K] INT8 codes, or null
  const float* sa;        // [r] INT8 per-channel scales
  const uint16_t* wg;     // [K] or null
  const uint16_t* W1;     // [h][r]
  const uint16_t* b1;     // [h]
  const uint16_t* W2;     // [r][h]
  const uint16_t* b2;     // [r]
  float b_g, alpha;
  int M, K, r, R1, R1p, h, gate;
  int P, ips;             // K-slices and iterations per slice
  int PG, tpg;            // row-tile groups and tiles per group
  int mode;               // EC_LAST, EC_GATHER or EC_RAW
  float* upart;           // EC_LAST/RAW: [ntb][P][16][R1] partial sums
  uint32_t* ctr;          // EC_LAST/RAW: [ntb] arrival counters
  float* v;               // [M][r] gated coordinates, fp32 (or null)
  uint16_t* vh;           // [M][vstride] act-dtype high part (or null)
  uint16_t* vl;           // [M][vstride] act-dtype low part  (or null)
  int vstride;
  float* u_out;           // EC_RAW: [M][R1]
  // fused: tagged words (tag << 32 | fp32 bits), kVCopies copies of
  //   EC_LAST:   v  [M][r]
  //   EC_GATHER: the slices' partial sums [P][M][R1]
  unsigned long long* vtag;
  unsigned long long* gen;  // fused: launch counters (see gen_increment)
  unsigned long long* ready;  // fused: kVCopies ready counters, kReadyStride apart
  int npub;                   // fused: publishers per launch
  int direct;                 // fused: consumers poll the tagged data itself
};

struct GemvParams {
  const uint32_t* qw;     // [N][K/8]
  const uint16_t* sc;     // [N][K/G] fp16 bits
  const uint8_t* zr;      // [N][K/G]
  const uint16_t* x;      // [M][K]
  uint16_t* y;            // [M][N]
  const uint16_t* B;      // [N][r] act dtype (null with INT8 B)
  const int8_t* B8;       // [N][r] INT8 codes, or null
  const float* sb;        // [N] INT8 per-channel scales
  const uint16_t* res;    // [M][N] residual added before the output's rounding, or null
  int M, N, K, G, ngroups, r;
  int S, ips, iw;         // K-slices per row group, iterations per slice and per wave
  int n_prod;             // EC workgroups at the head of the grid (fused)
  float* ypart;           // [S][M][N] partial sums (S > 1)
  float* eupart;          // EPI_LOCAL: [S][M][R1] partial sums of [A; w_g] x (S > 1)
  uint32_t* rb_ctr;       // [row groups] last-arriver counters
  int grid_total;         // fused: workgroups in the grid
  int wait_polls;
  int xlds;               // 1: the block's slice of x is staged in LDS
  int xstride;            // its LDS row stride in bytes
  int bpre;               // 1: the epilogue's rows of B are staged in LDS
  // LDS carve-up (byte offsets): [x | wave partials] [yacc] [EC u/hidden/v]
  // [rows of B] [gathered partials] [EC wave's result tiles] [scales];
  // EPI_LOCAL: the EC region holds u [16 MT][R1p] and v [16 MT][r]
  int lds_y, lds_e, lds_b, lds_g, lds_ev, lds_sz;
  int lds_a;              // EPI_LOCAL: [17][ips * 128 + 8] halves: A's 16 rows, w_g
  EcParams ec;
};

// Independent GEMV layer calls launched as one grid (up to kGroupMax of them,
// one kernel variant): member i owns workgroups [start[i], start[i+1]).
constexpr int kGroupMax = 4;
struct GemvGroup {
  GemvParams p[kGroupMax];
  int start[kGroupMax + 1];
  int n;
};

struct GemmParams {
  const uint32_t* qw;
  const uint16_t* sc;
  const uint8_t* zr;
  const uint16_t* x;
  uint16_t* y;
  const uint16_t* B;      // [N][r]
  const uint16_t* vh;     // [M][vstride]
  const uint16_t* vl;
  int M, N, K, G, ngroups, r, vstride;
  // split-K over S in {1, 2, 4, 8} K-slices (small tile grids): the slices'
  // fp32 tiles [S][tiles][128 x 128] (lane-major), tile counters, and with
  // EPI_LOCAL the slices' EC accumulators [S][tiles][4096] (lane-major)
  int S;
  float* ypart;
  uint32_t* ctr;
  float* epart;
  int tmw;                // token waves: 2 (128-token tiles) or 4 (256, EPI_NONE / EPI_READY)
  int roles;              // loading and multiplying waves (k_gemm_ws: tmw 4, S 1):
                          // 2 = 256 x 128 tiles, 3 = 256 x 256; else every wave both
  const uint16_t* res;    // [M][N] residual added before the output's rounding, or null
  // INT8 A and B (per-channel fp32 scales), or null: B8 for the
  // up-projection of EPI_READY / EPI_LOCAL_I8, A8 for EPI_LOCAL_I8
  const int8_t* A8;       // [r][K]
  const int8_t* B8;       // [N][r]
  const float* sa;        // [r]
  const float* sb;        // [N]
  // EPI_LOCAL (fully fused prefill): the projection's inputs
  const uint16_t* A;      // [r][K], r <= 16
  const uint16_t* wg;     // [K] (sigmoid gate) or null
  const uint16_t* W1;     // [h][r] (tanh-MLP gate) or null
  const uint16_t* b1;     // [h]
  const uint16_t* W2;     // [r][h]
  const uint16_t* b2;     // [r]
  float alpha, b_g;
  int gate, h;
};
// EPI_LOCAL GEMM: the EC stage tile holds A's 16 rows and w_g (row 16)
constexpr int kGemmEcRows = 17;

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Tokens per pass of the tanh-MLP gate in the local GEMV variant, whose LDS
// keeps 2048 floats for the gate's hidden layer (cap x h).
__host__ __device__ inline int local_tanh_cap(int M, int h) {
  const int c = 2048 / (h > 0 ? h : 1);
  return c < 1 ? 1 : (c < M ? c : M);
}
// Halves of the tanh-MLP gate's parameters (W1, b1, W2, b2) staged in LDS
// for the gate, or 0 when they exceed 4096 halves (then read from memory).
__host__ __device__ inline int tanh_stage_halves(int h, int r) {
  const int n = 2 * h * r + h + r;
  return n <= 4096 ? n : 0;
}

// GEMV workgroups have at most eight waves (a ninth would make the dispatcher
// reserve three waves' registers on every SIMD and halve residency); the EC
// variants give one of them to the EC wave.
constexpr int kGemvMaxThreads = 512;

// LDS of EC work: wave partials red [NW][kEcTiles][64][4] fp32, then
// u [16][R1p] fp32, hidden [h] fp32 and the v tile [16][r] fp32.
__host__ __device__ inline size_t ec_red_bytes(int NW) { return (size_t)NW * kEcTiles * 1024; }
__host__ __device__ inline size_t ec_lds_u_off() { return 0; }
__host__ __device__ inline size_t ec_lds_hid_off(int R1p) { return align_up((size_t)kTokTile * R1p * 4, 16); }
__host__ __device__ inline size_t ec_lds_v_off(int R1p, int h) { return ec_lds_hid_off(R1p) + align_up((size_t)h * 4, 16); }
__host__ __device__ inline size_t ec_lds_bytes(int R1p, int h, int r) {
  return ec_lds_v_off(R1p, h) + align_up((size_t)kTokTile * (r > 0 ? r : 1) * 4, 16);
}
// a producer workgroup: red, then the u/hidden/v region
__host__ __device__ inline size_t ec_block_lds(int NW, int R1p, int h, int r) {
  return ec_red_bytes(NW) + ec_lds_bytes(R1p, h, r);
}

// The kernels that read packed codes come in a 4-bit (_w4) and a 3-bit (_w3)
// build of spear_kernels.hip; the others only in the 4-bit one.
#define SPEAR_WEIGHT_LAUNCHERS(W)                                                                 \
  hipError_t launch_dequant_##W(int dt, const uint32_t* qw, const uint16_t* sc,                 \
                                const uint8_t* zr, uint16_t* out, int N, int K, int G,          \
                                hipStream_t st);                                                \
  hipError_t launch_gemv_##W(int dt, int MT, int RT, int epi, int nst, const GemvParams& p,     \
                             int grid, int block, size_t lds, hipStream_t st);                  \
  hipError_t launch_gemv_group_##W(int dt, int MT, int RT, int epi, const GemvGroup& g,         \
                                   int block, size_t lds, hipStream_t st);                      \
  hipError_t launch_gemm_##W(int dt, int epi, const GemmParams& p, hipStream_t st);
SPEAR_WEIGHT_LAUNCHERS(w4)
SPEAR_WEIGHT_LAUNCHERS(w3)
#undef SPEAR_WEIGHT_LAUNCHERS
hipError_t launch_ec(int dt, const EcParams& e, int grid, int block, int ipp, size_t lds,
                     hipStream_t st);
bool gemv_shape_supported(int MT, int RT);
hipError_t launch_gate(int dt, const EcParams& e, int ntb, size_t lds, hipStream_t st);
// y_norm[m] = RMSNorm(y[m]) * w (one workgroup per token row)
hipError_t launch_rmsnorm(int dt, const uint16_t* y, const uint16_t* w, float eps, uint16_t* y_norm,
                          int M, int N, hipStream_t st);
hipError_t launch_ec_up_acc(int dt, const float* v, const uint16_t* B, const int8_t* B8,
                            const float* sb, uint16_t* y, int M, int N, int r, hipStream_t st);

}  // namespace spear
