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
       EPI_FUSED = 2   // same, v produced by EC workgroups of the same grid
};

constexpr int kIterK = 128;      // K consumed per GEMV/EC iteration
constexpr int kTokTile = 16;     // tokens per MFMA token tile
constexpr int kGemmTM = 128;     // prefill tile: tokens
constexpr int kGemmTN = 128;     // prefill tile: output rows
constexpr int kGemmTK = 64;      // prefill tile: K per stage
constexpr int kGemmLdsRow = kGemmTK + 8;  // padded LDS row (halves)
constexpr int kVCopies = 8;      // tagged EC-coordinate copies (one per XCD)

// Workspace: a fixed counter block at the start, shared by every kind of call
// (each call returns its counters to zero), then the call's data regions.
constexpr size_t kCounterBytes = 65536;
constexpr size_t kCtrGen = 0;        // launch generation of the fused path
constexpr size_t kCtrDone = 4;       // fused grid: blocks done
constexpr size_t kCtrEc = 256;       // EC-slice counters, one per token tile
constexpr int kMaxEcCounters = 64;
constexpr size_t kCtrRows = 512;     // split-K counters, one per row group
constexpr int kMaxRowCounters = (int)((kCounterBytes - kCtrRows) / 4);

// Tag of the EC coordinates published by the fused launch of generation g:
// a multiplicative hash, so that leftover data of another call is never
// mistaken for a current coordinate (2^-32 chance per word).
__host__ __device__ inline uint32_t ec_tag(uint32_t gen) { return ((gen + 1u) * 0x9E3779B1u) | 1u; }

// EC projection / gate work of one token tile (16 tokens) and one K-slice.
struct EcParams {
  const uint16_t* x;      // [M][K]
  const uint16_t* A;      // [r][K]
  const uint16_t* wg;     // [K] or null
  const uint16_t* W1;     // [h][r]
  const uint16_t* b1;     // [h]
  const uint16_t* W2;     // [r][h]
  const uint16_t* b2;     // [r]
  float b_g, alpha;
  int M, K, r, R1, R1p, h, gate;
  int P, ips;             // K-slices and 128-wide iterations per slice
  int raw;                // 1: store u = [A; w_g] x only (no gate)
  float* upart;           // [ntb][P][16][R1] partial sums (P > 1)
  uint32_t* ctr;          // [ntb] last-arriver counters
  float* v;               // [M][r] gated coordinates, fp32
  uint16_t* vh;           // [M][vstride] act-dtype high part (or null)
  uint16_t* vl;           // [M][vstride] act-dtype low part  (or null)
  int vstride;
  float* u_out;           // raw mode: [M][R1]
  unsigned long long* vtag;  // fused: [kVCopies][M][r] (tag << 32 | fp32 bits)
  uint32_t* gen;          // fused: launch generation (tag = ec_tag(gen))
  uint32_t epoch;
};

struct GemvParams {
  const uint32_t* qw;     // [N][K/8]
  const uint16_t* sc;     // [N][K/G] fp16 bits
  const uint8_t* zr;      // [N][K/G]
  const uint16_t* x;      // [M][K]
  uint16_t* y;            // [M][N]
  const uint16_t* B;      // [N][r]
  int M, N, K, G, ngroups, r;
  int S, ips, iw;         // K-slices per row group, iterations per slice and per wave
  int n_prod;             // EC workgroups at the head of the grid (fused)
  float* ypart;           // [S][M][N] partial sums (S > 1)
  uint32_t* rb_ctr;       // [row tiles] last-arriver counters
  uint32_t* done_ctr;     // fused: arrivals of every workgroup of the grid
  int grid_total;              // fused: workgroups in the grid
  int wait_polls;
  uint32_t epoch;
  EcParams ec;
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
};

__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// LDS carve-up of an EC block: u [16][R1p] fp32, hidden [h] fp32, v tile [16][r] fp32.
__host__ __device__ inline size_t ec_lds_u_off() { return 0; }
__host__ __device__ inline size_t ec_lds_hid_off(int R1p) { return align_up((size_t)kTokTile * R1p * 4, 16); }
__host__ __device__ inline size_t ec_lds_v_off(int R1p, int h) { return ec_lds_hid_off(R1p) + align_up((size_t)h * 4, 16); }
__host__ __device__ inline size_t ec_lds_bytes(int R1p, int h, int r) {
  return ec_lds_v_off(R1p, h) + align_up((size_t)kTokTile * (r > 0 ? r : 1) * 4, 16);
}

// LDS carve-up of a GEMV block of NW waves and RT row tiles:
//   red:  per-wave partial tiles, NW x RT x MT x 1 KB
//   yacc: the block's sums [16*MT tokens][16*RT rows] fp32
//   E:    an EC block (v tile for the epilogue; u/hidden for the fallback),
//         then the epilogue's rows of B
__host__ __device__ inline size_t gemv_lds_y_off(int NW, int RT, int MT) {
  return (size_t)NW * RT * MT * 1024;
}
__host__ __device__ inline size_t gemv_lds_e_off(int NW, int RT, int MT) {
  return gemv_lds_y_off(NW, RT, MT) + (size_t)RT * MT * 1024;
}
// after E (and B, when the EC is on): the staged scales/zero points
// [16*RT rows][groups of the block's K-slice] as u32
__host__ __device__ inline size_t gemv_lds_sz_off(int NW, int RT, int MT, int R1p, int h, int r,
                                                  bool ec) {
  size_t o = gemv_lds_e_off(NW, RT, MT);
  if (ec) o += ec_lds_bytes(R1p, h, r) + align_up((size_t)16 * RT * r * 2, 16);
  return align_up(o, 16);
}

hipError_t launch_dequant(int dt, const uint32_t* qw, const uint16_t* sc, const uint8_t* zr,
                          uint16_t* out, int N, int K, int G, hipStream_t st);
hipError_t launch_ec(int dt, const EcParams& e, int ntb, int block, size_t lds, hipStream_t st);
bool gemv_shape_supported(int MT, int RT);
hipError_t launch_gemv(int dt, int MT, int RT, int epi, const GemvParams& p, int grid, int block,
                       size_t lds, hipStream_t st);
hipError_t launch_gemm(int dt, int epi, const GemmParams& p, hipStream_t st);
hipError_t launch_gate(int dt, const EcParams& e, int ntb, size_t lds, hipStream_t st);
hipError_t launch_ec_up_acc(int dt, const float* v, const uint16_t* B, uint16_t* y, int M,
                            int N, int r, hipStream_t st);

}  // namespace spear
