// gfx950 (MI355X) kernels of the W4+EC linear layer.
//
// Y = X . What^T + alpha * (gate (.) (X . A^T)) . B^T      (SPEAR, section 3.1, Eq. 3)
// What[n][k] = (q[n][k] - z[n][k/G]) * s[n][k/G]          (sections 3.2, 5.1)
//
// MFMA operand convention (v_mfma_f32_16x16x32_{f16,bf16}, wave64): lane l
// supplies row (l % 16) of the A operand and column (l % 16) of the B operand,
// each as 8 consecutive K positions of K-block (l / 16); the 16x16 fp32 result
// gives lane l the column (l % 16) and rows 4*(l/16) .. 4*(l/16)+3. Any
// permutation of the K positions is harmless as long as both operands use it.
//
// Kernels:
//   k_dequant  bit-exact dequantisation diagnostic
//   k_ec       EC projection u = [A; w_g] x over a K-slice, last-arriver
//              reduction across slices, gate, v = alpha * gate (.) u
//   k_gemv     decode: 4-bit product with MFMA on one 16-row tile per block,
//              per-128 dequant correction, cross-wave (and, for long K,
//              cross-block) reduction, epilogue adding B v; in the fused
//              variant the grid's first blocks run k_ec's work and publish v
//              as tagged words that the other blocks poll
//   k_gemm     prefill: LDS-tiled 4-bit GEMM (dequantised tiles, double
//              buffered), MFMA epilogue adding B v from the EC pre-kernel
//   k_gate, k_ec_up_acc   the naive split chain's separate gate and
//              reprojection+accumulate launches
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "spear_internal.h"

namespace spear {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

template <int DT>
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  if constexpr (DT == DT_F16)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <int DT>
__device__ __forceinline__ float act2f(uint32_t bits16) {
  if constexpr (DT == DT_F16)
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
  else
    return __uint_as_float(bits16 << 16);
}

// Round-to-nearest-even conversion to the activation dtype.
template <int DT>
__device__ __forceinline__ uint16_t f2act(float f) {
  if constexpr (DT == DT_F16)
    return __builtin_bit_cast(uint16_t, (_Float16)f);
  else
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }

// Codes of one packed word as biased act-dtype values, paired (q0,q4),
// (q1,q5), (q2,q6), (q3,q7). OR-ing a 4-bit code into the mantissa of
// 1024.0 (fp16 0x6400) or 128.0 (bf16 0x4300) gives exactly 1024+q / 128+q.
template <int DT>
__device__ __forceinline__ u32x4 unpack_biased(uint32_t w) {
  constexpr uint32_t kMag = DT == DT_F16 ? 0x64006400u : 0x43004300u;
  u32x4 r;
  r[0] = (w & 0x000F000Fu) | kMag;
  r[1] = ((w >> 4) & 0x000F000Fu) | kMag;
  r[2] = ((w >> 8) & 0x000F000Fu) | kMag;
  r[3] = ((w >> 12) & 0x000F000Fu) | kMag;
  return r;
}
// Same, with the mask and the magic number in registers (`km` = 0x000F000F,
// `kg` = the magic pair): each code pair is then one v_and_or_b32 (plus a
// shift), which the literal-constant form above does not compile to.
__device__ __forceinline__ u32x4 unpack_biased_r(uint32_t w, uint32_t km, uint32_t kg) {
  u32x4 r;
  r[0] = (w & km) | kg;
  r[1] = ((w >> 4) & km) | kg;
  r[2] = ((w >> 8) & km) | kg;
  r[3] = ((w >> 12) & km) | kg;
  return r;
}
// Opaque copy of a constant in a VGPR (the compiler cannot fold it back into
// an instruction literal).
__device__ __forceinline__ uint32_t opaque_v(uint32_t c) {
  asm volatile("" : "+v"(c));
  return c;
}
template <int DT>
__device__ __forceinline__ constexpr float code_bias() { return DT == DT_F16 ? 1024.f : 128.f; }

// Reorder 8 consecutive activations (x0..x7) into the pairing above.
__device__ __forceinline__ u32x4 pair_like_codes(u32x4 x) {
  u32x4 r;
  r[0] = (x[0] & 0xFFFFu) | (x[2] << 16);
  r[1] = (x[0] >> 16) | (x[2] & 0xFFFF0000u);
  r[2] = (x[1] & 0xFFFFu) | (x[3] << 16);
  r[3] = (x[1] >> 16) | (x[3] & 0xFFFF0000u);
  return r;
}

template <int DT>
__device__ __forceinline__ u32x4 ones8() {
  constexpr uint32_t o = DT == DT_F16 ? 0x3C003C00u : 0x3F803F80u;
  return u32x4{o, o, o, o};
}

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *(const u32x4*)p; }

// Raw buffer loads through a bounds-checked resource (gfx9 descriptor word 3
// = 0x00020000): a byte offset at or past `bytes` reads as zero. Masked
// elements are given the offset kOOB, so every load is issued without a
// branch and a wave's loads all stay in flight together.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr uint32_t kOOB = 0x80000000u;
__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4 bld128(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
// voffset (per lane, carries the mask) + soffset (wave-uniform)
__device__ __forceinline__ u32x4 bld128s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t bld16s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t bld8s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b8(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t bld16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}
__device__ __forceinline__ uint32_t bld8(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b8(r, off, 0, 0);
}

// Cross-workgroup data (partial sums, the EC coordinates, flags, counters)
// moves only through relaxed agent-scope atomic accesses: on gfx950 these are
// plain loads/stores with the sc1 bit, coherent across the eight XCDs' L2s on
// every access, so no cache-wide writeback or invalidate is ever issued.
// Ordering comes from waiting for the stores to complete (s_waitcnt) before
// the barrier that precedes the publishing atomic.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent_u32(const uint32_t* p) {
  return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// All of this thread's memory operations have completed; then the block meets.
__device__ __forceinline__ void complete_and_sync() {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
}

// Last-arriver detection: one relaxed agent-scope fetch-add per arrival (no
// compare-and-swap retries, which serialise at one memory round trip each).
// The arrival that completes `total` resets the counter to zero, so every
// launch (also a replayed graph) starts from zero; the workspace holding the
// counters is zero-filled once before first use. Callers publish their data
// with st_agent and complete_and_sync() before arriving, and the last arriver
// reads it back with ld_agent.
__device__ __forceinline__ bool arrive_last(uint32_t* ctr, uint32_t total) {
  const uint32_t old = __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (old + 1u != total) return false;
  __hip_atomic_store(ctr, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// ---------------------------------------------------------------------------
// Dequantisation diagnostic: one thread per packed word, eight outputs.
// (q - z) * s is exact in fp32 (<= 4 + 11 significant bits); the single
// rounding is the conversion to the activation dtype.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void k_dequant(const uint32_t* __restrict__ qw,
                                                 const uint16_t* __restrict__ sc,
                                                 const uint8_t* __restrict__ zr,
                                                 uint16_t* __restrict__ out, int N, int K, int G) {
  const int kw = K >> 3;
  const long long nwords = (long long)N * kw;
  const long long wi = (long long)blockIdx.x * 256 + threadIdx.x;
  if (wi >= nwords) return;
  const int n = (int)(wi / kw);
  const int k = (int)(wi % kw) * 8;
  const int ng = K / G;
  const int g = k / G;
  const float s = h2f(sc[(long long)n * ng + g]);
  const int z = zr[(long long)n * ng + g];
  const uint32_t w = qw[wi];
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q0 = (w >> (8 * i)) & 15, q1 = (w >> (8 * i + 4)) & 15;
    const uint32_t lo = f2act<DT>((float)(q0 - z) * s);
    const uint32_t hi = f2act<DT>((float)(q1 - z) * s);
    o[i] = lo | (hi << 16);
  }
  *(u32x4*)(out + (long long)n * K + k) = u32x4{o[0], o[1], o[2], o[3]};
}

// ---------------------------------------------------------------------------
// EC projection of one token tile over iterations [it_beg, it_end):
// u_lds[t][j] = sum_k x[16*tb + t][k] * R[j][k], R = [A; w_g] (R1 rows), as a
// sum over the block's waves in a fixed order (wave 0 first).
// ---------------------------------------------------------------------------
// Row tiles of [A; w_g] projected together (bounds the registers the
// two-iteration load batch needs).
constexpr int kEcTiles = 2;

template <int DT>
__device__ void ec_project_tile(const EcParams& e, int tb, int it_beg, int it_end, float* u_lds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int NW = blockDim.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int m = tb * kTokTile + lr;
  const int RTe = (e.R1 + 15) >> 4;
  const rsrc_t rx = make_rsrc(e.x, (uint32_t)e.M * e.K * 2);
  const rsrc_t ra = make_rsrc(e.A, (uint32_t)e.r * e.K * 2);
  const rsrc_t rg = make_rsrc(e.wg, e.gate == GATE_SIGMOID ? (uint32_t)e.K * 2 : 0u);
  const uint32_t xoff = m < e.M ? (uint32_t)m * e.K * 2 + 64 * lg : kOOB;
  for (int tg0 = 0; tg0 < RTe; tg0 += kEcTiles) {
    const int nt = min(kEcTiles, RTe - tg0);
    f32x4 acc[kEcTiles];
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint32_t aoff[kEcTiles], goff[kEcTiles];
    bool has_g[kEcTiles];
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t) {
      const int j = (tg0 + t) * 16 + lr;
      aoff[t] = j < e.r ? (uint32_t)j * e.K * 2 + 64 * lg : kOOB;
      goff[t] = (j == e.r && e.gate == GATE_SIGMOID) ? 64u * lg : kOOB;
      // uniform: does this row tile hold the gate row w_g?
      has_g[t] = e.gate == GATE_SIGMOID && e.r >= (tg0 + t) * 16 && e.r < (tg0 + t + 1) * 16;
    }
    // two iterations per pass with all of their loads issued first
    for (int it = it_beg + wave; it < it_end; it += 2 * NW) {
      const int it2 = it + NW;
      const uint32_t kb = (uint32_t)it * (kIterK * 2);
      const uint32_t kb2 = (uint32_t)it2 * (kIterK * 2);
      const bool ok2 = it2 < it_end;
      u32x4 xv[2][4], av[2][kEcTiles][4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        xv[0][jj] = bld128(rx, xoff + kb + 16 * jj);
        xv[1][jj] = bld128(rx, ok2 ? xoff + kb2 + 16 * jj : kOOB);
      }
#pragma unroll
      for (int t = 0; t < kEcTiles; ++t) {
        if (t < nt) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            av[0][t][jj] = bld128(ra, aoff[t] + kb + 16 * jj);
            av[1][t][jj] = bld128(ra, ok2 ? aoff[t] + kb2 + 16 * jj : kOOB);
            if (has_g[t]) {
              av[0][t][jj] |= bld128(rg, goff[t] + kb + 16 * jj);
              av[1][t][jj] |= bld128(rg, ok2 ? goff[t] + kb2 + 16 * jj : kOOB);
            }
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int t = 0; t < kEcTiles; ++t)
          if (t < nt)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) acc[t] = mfma16<DT>(av[h][t][jj], xv[h][jj], acc[t]);
    }
    // deterministic cross-wave sum: wave 0 stores, waves 1.. add in order
    for (int w = 0; w < NW; ++w) {
      __syncthreads();
      if (wave == w) {
#pragma unroll
        for (int t = 0; t < kEcTiles; ++t) {
          if (t < nt) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int j = (tg0 + t) * 16 + 4 * lg + i;
              float* dst = u_lds + lr * e.R1p + j;
              *dst = (w == 0) ? acc[t][i] : *dst + acc[t][i];
            }
          }
        }
      }
    }
    __syncthreads();
  }
}

// Gate of one token tile: from u (LDS, [16][R1p]) to v_tile (LDS, [16][r]):
// v = alpha * g * u (sigmoid-linear), alpha * (1 + tanh(W2 ReLU(W1 u + b1) + b2)) (.) u
// (tanh-MLP), or alpha * u (gate one).
template <int DT>
__device__ void ec_gate_tile(const EcParams& e, int cnt, const float* u_lds, float* hid,
                             float* v_tile) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int r = e.r;
  if (e.gate == GATE_TANH) {
    for (int t = 0; t < cnt; ++t) {
      const float* u = u_lds + t * e.R1p;
      for (int i = tid; i < e.h; i += nthr) {
        float a = act2f<DT>(e.b1[i]);
        const uint16_t* w1 = e.W1 + (size_t)i * r;
        for (int j = 0; j < r; ++j) a += act2f<DT>(w1[j]) * u[j];
        hid[i] = a > 0.f ? a : 0.f;
      }
      __syncthreads();
      for (int j = tid; j < r; j += nthr) {
        float a = act2f<DT>(e.b2[j]);
        const uint16_t* w2 = e.W2 + (size_t)j * e.h;
        for (int i = 0; i < e.h; ++i) a += act2f<DT>(w2[i]) * hid[i];
        v_tile[t * r + j] = e.alpha * (1.f + tanhf(a)) * u[j];
      }
      __syncthreads();
    }
  } else {
    for (int idx = tid; idx < cnt * r; idx += nthr) {
      const int t = idx / r, j = idx - t * r;
      float g = 1.f;
      if (e.gate == GATE_SIGMOID) {
        const float z = u_lds[t * e.R1p + r] + e.b_g;
        g = z >= 0.f ? 1.f / (1.f + __expf(-z)) : __expf(z) / (1.f + __expf(z));
      }
      v_tile[idx] = e.alpha * g * u_lds[t * e.R1p + j];
    }
    __syncthreads();
  }
}

// One EC block: token tile tb, K-slice p. Projects, reduces across slices
// (last arriver), applies the gate and publishes v: as fp32 (consumed by a
// later kernel), as act-dtype hi/lo parts (the GEMM epilogue), and/or as
// tagged 64-bit words (tag << 32 | fp32 bits) in one copy per XCD, which the
// fused kernel's workgroups poll: a word is current when its tag matches.
template <int DT>
__device__ void ec_block(const EcParams& e, int tb, int p, char* smem) {
  __shared__ int s_last;
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int IT = e.K / kIterK;
  const int it_beg = p * e.ips, it_end = min(IT, it_beg + e.ips);
  float* u_lds = (float*)(smem + ec_lds_u_off());
  float* hid = (float*)(smem + ec_lds_hid_off(e.R1p));
  float* v_tile = (float*)(smem + ec_lds_v_off(e.R1p, e.h));
  const int m0 = tb * kTokTile;
  const int cnt = min(kTokTile, e.M - m0);

  ec_project_tile<DT>(e, tb, it_beg, it_end, u_lds);

  if (e.P > 1) {
    float* part = e.upart + ((size_t)tb * e.P + p) * kTokTile * e.R1;
    for (int idx = tid; idx < cnt * e.R1; idx += nthr) {
      const int t = idx / e.R1, j = idx - t * e.R1;
      st_agent(part + idx, u_lds[t * e.R1p + j]);
    }
    complete_and_sync();
    if (tid == 0) s_last = arrive_last(e.ctr + tb, (uint32_t)e.P) ? 1 : 0;
    __syncthreads();
    if (!s_last) return;
    const float* base = e.upart + (size_t)tb * e.P * kTokTile * e.R1;
    for (int idx = tid; idx < cnt * e.R1; idx += nthr) {
      float a = 0.f;
      for (int q = 0; q < e.P; ++q) a += ld_agent(base + (size_t)q * kTokTile * e.R1 + idx);
      const int t = idx / e.R1, j = idx - t * e.R1;
      u_lds[t * e.R1p + j] = a;
    }
    __syncthreads();
  }

  if (e.raw) {
    for (int idx = tid; idx < cnt * e.R1; idx += nthr) {
      const int t = idx / e.R1, j = idx - t * e.R1;
      e.u_out[(size_t)(m0 + t) * e.R1 + j] = u_lds[t * e.R1p + j];
    }
    return;
  }

  ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
  if (e.v)
    for (int idx = tid; idx < cnt * e.r; idx += nthr) e.v[(size_t)m0 * e.r + idx] = v_tile[idx];
  if (e.vh) {
    for (int idx = tid; idx < cnt * e.vstride; idx += nthr) {
      const int t = idx / e.vstride, j = idx - t * e.vstride;
      float val = j < e.r ? v_tile[t * e.r + j] : 0.f;
      const uint16_t hi = f2act<DT>(val);
      const uint16_t lo = f2act<DT>(val - act2f<DT>(hi));
      e.vh[(size_t)(m0 + t) * e.vstride + j] = hi;
      e.vl[(size_t)(m0 + t) * e.vstride + j] = lo;
    }
  }
  if (e.vtag) {
    const uint32_t tag = ec_tag(ld_agent_u32(e.gen));
    const size_t per_copy = (size_t)e.M * e.r;
    for (int idx = tid; idx < cnt * e.r * kVCopies; idx += nthr) {
      const int c = idx / (cnt * e.r), o = idx - c * (cnt * e.r);
      const unsigned long long w =
          ((unsigned long long)tag << 32) | __float_as_uint(v_tile[o]);
      __hip_atomic_store(e.vtag + c * per_copy + (size_t)m0 * e.r + o, w, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int DT>
__global__ __launch_bounds__(512) void k_ec(EcParams e) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  ec_block<DT>(e, blockIdx.x / e.P, blockIdx.x % e.P, smem);
}

// Naive chain, gate launch: reads u [M][R1] and writes v [M][r].
template <int DT>
__global__ __launch_bounds__(256) void k_gate(EcParams e) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  float* u_lds = (float*)(smem + ec_lds_u_off());
  float* hid = (float*)(smem + ec_lds_hid_off(e.R1p));
  float* v_tile = (float*)(smem + ec_lds_v_off(e.R1p, e.h));
  const int m0 = blockIdx.x * kTokTile;
  const int cnt = min(kTokTile, e.M - m0);
  for (int idx = threadIdx.x; idx < cnt * e.R1; idx += blockDim.x) {
    const int t = idx / e.R1, j = idx - t * e.R1;
    u_lds[t * e.R1p + j] = e.u_out[(size_t)(m0 + t) * e.R1 + j];
  }
  __syncthreads();
  ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
  for (int idx = threadIdx.x; idx < cnt * e.r; idx += blockDim.x) e.v[(size_t)m0 * e.r + idx] = v_tile[idx];
}

// Naive chain, reprojection + accumulate: y[m][n] += sum_j v[m][j] B[n][j].
template <int DT>
__global__ __launch_bounds__(256) void k_ec_up_acc(const float* __restrict__ v,
                                                   const uint16_t* __restrict__ B,
                                                   uint16_t* __restrict__ y, int M, int N, int r) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  float a = act2f<DT>(y[idx]);
  for (int j = 0; j < r; ++j) a += v[(size_t)m * r + j] * act2f<DT>(B[(size_t)n * r + j]);
  y[idx] = f2act<DT>(a);
}

// Every block of the fused grid arrives here once when it is done; the last
// one advances the generation that tags the next launch's EC coordinates, so
// that a replayed graph (same epoch) never reads the previous replay's values.
__device__ __forceinline__ void fused_exit(const GemvParams& a, uint32_t gen) {
  complete_and_sync();
  if (threadIdx.x == 0 && arrive_last(a.done_ctr, (uint32_t)a.grid_total))
    __hip_atomic_store(a.ec.gen, gen + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// Decode GEMV. A block owns RT row tiles (16 rows each) and a K-slice of
// iterations (128 K each); each of its NW waves walks a contiguous chunk of
// that slice as a software pipeline: the codes, scales, zero points and
// activation fragments of iteration it+1 are in flight while iteration it is
// computed, so memory and compute overlap within every wave. The MFMA
// multiplies activations (A operand, 16 token rows) by the biased codes (B
// operand, 16 weight rows as columns), so each lane owns one weight row per
// tile and needs one scale and one zero point per iteration:
//   sum_k x (q - z) s = s * ( sum_k x (bias + q) - (bias + z) * sum_k x ),
// with sum_k x from an MFMA against ones, shared by the RT tiles. Waves are
// reduced in LDS in a fixed order; K-slices through partial sums and a last
// arriver.
//
// Fused variant: the first n_prod blocks of the grid are EC blocks (above).
// The others, after their main loop, poll the tagged EC coordinates of their
// XCD copy (bounded; on time-out they compute the EC themselves) and add
// B v in the epilogue. Every block arrives at a done counter at its end; the
// last one advances the generation that tags the next launch's coordinates.
// ---------------------------------------------------------------------------
template <int DT, int MT, int RT, int EPI>
__global__ __launch_bounds__(512) void k_gemv(GemvParams a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int s_flag;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int NW = blockDim.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  int bid = blockIdx.x;
  uint32_t gen = 0;
  if constexpr (EPI == EPI_FUSED) {
    gen = ld_agent_u32(a.ec.gen);
    if (bid < a.n_prod) {
      ec_block<DT>(a.ec, bid / a.ec.P, bid % a.ec.P, smem);
      fused_exit(a, gen);
      return;
    }
    bid -= a.n_prod;
  }
  constexpr int RB = 16 * RT;
  const int M = a.M, N = a.N, K = a.K, G = a.G;
  const int IT = K / kIterK;
  const int rg = bid / a.S, s = bid - (bid / a.S) * a.S;
  const int n0 = rg * RB;
  const int it_blk = s * a.ips;
  const int it_end = min(IT, it_blk + a.ips);
  const int iw_beg = it_blk + wave * a.iw;
  const int iw_end = min(it_end, iw_beg + a.iw);

  const rsrc_t rq = make_rsrc(a.qw, (uint32_t)N * (K / 2));
  const rsrc_t rsc = make_rsrc(a.sc, (uint32_t)N * a.ngroups * 2);
  const rsrc_t rz = make_rsrc(a.zr, (uint32_t)N * a.ngroups);
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)M * K * 2);

  // the EC epilogue's rows of B ([16*RT][r], fp16/bf16) are fetched up front
  // when r is a multiple of 8 and two 16-byte chunks per thread cover them;
  // otherwise the epilogue reads B directly
  constexpr int BCH = 2;
  const int r = a.r;
  const int bchunks = EPI != EPI_NONE && (r & 7) == 0 ? RB * r / 8 : 0;
  const bool bpre = bchunks > 0 && bchunks <= BCH * (int)blockDim.x;
  u32x4 bst[BCH];
  if (bpre) {
    const rsrc_t rb = make_rsrc(a.B, (uint32_t)N * r * 2);
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int ci = tid + c * (int)blockDim.x;
      bst[c] = bld128(rb, ci < bchunks ? (uint32_t)n0 * r * 2 + 16u * ci : kOOB);
    }
  }

  // one batch = one 128-wide iteration of every row tile: codes, scales,
  // zero points and the activation fragments. The per-lane part of every
  // offset (row, token, lane group; kOOB for rows >= N or tokens >= M) is
  // fixed for the whole loop; the iteration enters as a wave-uniform soffset.
  uint32_t vw[RT], vx[MT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int n = n0 + 16 * t + lr;
    vw[t] = n < N ? (uint32_t)n * (K / 2) + 16 * lg : kOOB;
  }
  // lanes of tokens >= M read the last token's row: their MFMA rows only feed
  // outputs that are never stored, and in-bounds duplicate addresses are far
  // cheaper for the address unit than masked (out-of-range) lanes
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = min(16 * mt + lr, M - 1);
    vx[mt] = ((uint32_t)m * K + 32 * lg) * 2;
  }
  auto load = [&](u32x4 (&w)[RT], u32x4 (&xv)[MT][4], int it) {
#pragma unroll
    for (int t = 0; t < RT; ++t) w[t] = bld128s(rq, vw[t], (uint32_t)it * (kIterK / 2));
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        xv[mt][jj] = bld128s(rx, vx[mt] + 16 * jj, (uint32_t)it * (kIterK * 2));
  };

  // scales and zero points of the block's rows and groups, staged once in
  // LDS with coalesced loads ([row][group] as s | z << 16): per-iteration
  // scattered 2- and 1-byte loads would cost a cache-line request per row
  const int ipg = G / kIterK;  // iterations per quantisation group
  const int g_lo = it_blk / ipg;
  const int ngb = (it_end - 1) / ipg + 1 - g_lo;
  const int ngs = ngb | 1;  // odd LDS row stride: rows fall on distinct banks
  uint32_t* szs = (uint32_t*)(smem + gemv_lds_sz_off(NW, RT, MT, a.ec.R1p, a.ec.h, r, EPI != EPI_NONE));
  // the first batch goes out before the staging loads so that both overlap
  u32x4 wA[RT], wB[RT];
  u32x4 xA[MT][4], xB[MT][4];
  if (iw_beg < iw_end) load(wA, xA, iw_beg);
  for (int idx = tid; idx < RB * ngb; idx += blockDim.x) {
    const int row = idx / ngb, gg = idx - row * ngb;
    const int n = n0 + row;
    const uint32_t e = (uint32_t)n * a.ngroups + g_lo + gg;
    const uint32_t sv = bld16(rsc, n < N ? e * 2 : kOOB);
    const uint32_t zv = bld8(rz, n < N ? e : kOOB);
    szs[row * ngs + gg] = sv | (zv << 16);
  }
  __syncthreads();
  constexpr float kBias = code_bias<DT>();
  f32x4 acc[RT][MT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint32_t km = opaque_v(0x000F000Fu);
  const uint32_t kg = opaque_v(DT == DT_F16 ? 0x64006400u : 0x43004300u);
  auto compute = [&](const u32x4 (&w)[RT], const u32x4 (&xv)[MT][4], int it) {
    f32x4 xb[MT];
    u32x4 xp[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      xb[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        xb[mt] = mfma16<DT>(xv[mt][jj], ones8<DT>(), xb[mt]);
        xp[mt][jj] = pair_like_codes(xv[mt][jj]);
      }
    }
    const int gg = it / ipg - g_lo;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      u32x4 wd[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) wd[jj] = unpack_biased_r(w[t][jj], km, kg);
      const uint32_t sz = szs[(16 * t + lr) * ngs + gg];
      const float sf = h2f((uint16_t)(sz & 0xFFFF));
      const float cf = kBias + (float)(sz >> 16);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 pacc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) pacc = mfma16<DT>(xp[mt][jj], wd[jj], pacc);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[t][mt][i] += sf * (pacc[i] - cf * xb[mt][i]);
      }
    }
  };

  // software pipeline over this wave's iterations: batch it+1 is in flight
  // while batch it is computed (two register sets, alternating). Loads past
  // the wave's last iteration re-read that iteration (never computed), so
  // every load is unconditional.
  if (iw_beg < iw_end) {
    const int last = iw_end - 1;
    for (int it = iw_beg; it < iw_end; it += 2) {
      load(wB, xB, min(it + 1, last));
      __builtin_amdgcn_sched_barrier(0);
      compute(wA, xA, it);
      if (it + 1 >= iw_end) break;
      load(wA, xA, min(it + 2, last));
      __builtin_amdgcn_sched_barrier(0);
      compute(wB, xB, it + 1);
    }
  }

  // ---- cross-wave reduction (fixed order) into yacc[token][row]
  float* red = (float*)smem;
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
      *(f32x4*)(red + (((wave * RT + t) * MT + mt) * 64 + lane) * 4) = acc[t][mt];
  __syncthreads();
  float* yacc = (float*)(smem + gemv_lds_y_off(NW, RT, MT));
  constexpr int YS = RB;  // yacc row stride: [token][RB rows]
  for (int e = tid; e < 256 * RT * MT; e += blockDim.x) {
    const int tm = e >> 8, rem = e & 255, ln = rem >> 2, i = rem & 3;
    const int t = tm / MT, mt = tm - t * MT;
    float v = 0.f;
    for (int w = 0; w < NW; ++w) v += red[(((w * RT + t) * MT + mt) * 64 + ln) * 4 + i];
    const int tok = 16 * mt + 4 * (ln >> 4) + i, row = 16 * t + (ln & 15);
    yacc[tok * YS + row] = v;
  }
  __syncthreads();

  // ---- cross-block split-K reduction: last arriver sums the slices in order
  if (a.S > 1) {
    for (int e = tid; e < RB * M; e += blockDim.x) {
      const int m = e / RB, row = e - m * RB;
      if (n0 + row < N) st_agent(a.ypart + ((size_t)s * M + m) * N + n0 + row, yacc[m * YS + row]);
    }
    complete_and_sync();
    if (tid == 0) s_flag = arrive_last(a.rb_ctr + rg, (uint32_t)a.S) ? 1 : 0;
    __syncthreads();
    if (!s_flag) {
      if constexpr (EPI == EPI_FUSED) fused_exit(a, gen);
      return;
    }
    for (int e = tid; e < RB * M; e += blockDim.x) {
      const int m = e / RB, row = e - m * RB;
      if (n0 + row < N) {
        float v = 0.f;
        for (int q = 0; q < a.S; ++q) v += ld_agent(a.ypart + ((size_t)q * M + m) * N + n0 + row);
        yacc[m * YS + row] = v;
      }
    }
    __syncthreads();
  }

  if constexpr (EPI == EPI_NONE) {
    for (int e = tid; e < RB * M; e += blockDim.x) {
      const int m = e / RB, row = e - m * RB;
      if (n0 + row < N) a.y[(size_t)m * N + n0 + row] = f2act<DT>(yacc[m * YS + row]);
    }
  } else {
    const EcParams& e = a.ec;
    char* ec_smem = smem + gemv_lds_e_off(NW, RT, MT);
    float* v_tile = (float*)(ec_smem + ec_lds_v_off(e.R1p, e.h));
    uint16_t* bs = (uint16_t*)(ec_smem + ec_lds_bytes(e.R1p, e.h, r));  // [RB][r]
    if (bpre) {
#pragma unroll
      for (int c = 0; c < BCH; ++c) {
        const int ci = tid + c * (int)blockDim.x;
        if (ci < bchunks) *(u32x4*)(bs + 8 * ci) = bst[c];
      }
      __syncthreads();
    }
    const int ntb = (M + kTokTile - 1) / kTokTile;
    const uint32_t tag = ec_tag(gen);
    const unsigned long long* vcopy =
        e.vtag ? e.vtag + (size_t)(blockIdx.x % kVCopies) * ((size_t)M * r) : nullptr;
    for (int tb = 0; tb < ntb; ++tb) {
      const int m0 = tb * kTokTile, cnt = min(kTokTile, M - m0);
      bool have = true;
      if constexpr (EPI == EPI_FUSED) {
        // bounded poll of the tagged coordinates; every thread checks its share
        for (int poll = 0;; ++poll) {
          int stale = 0;
          for (int idx = tid; idx < cnt * r; idx += blockDim.x) {
            const unsigned long long w = __hip_atomic_load(
                const_cast<unsigned long long*>(vcopy) + (size_t)m0 * r + idx, __ATOMIC_RELAXED,
                __HIP_MEMORY_SCOPE_AGENT);
            if ((uint32_t)(w >> 32) != tag) stale = 1;
            else v_tile[idx] = __uint_as_float((uint32_t)w);
          }
          if (!__syncthreads_or(stale)) break;
          if (poll >= a.wait_polls) { have = false; break; }
          __builtin_amdgcn_s_sleep(2);
        }
        if (!have) {
          float* u_lds = (float*)(ec_smem + ec_lds_u_off());
          float* hid = (float*)(ec_smem + ec_lds_hid_off(e.R1p));
          ec_project_tile<DT>(e, tb, 0, IT, u_lds);
          ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
        }
      } else {
        for (int idx = tid; idx < cnt * r; idx += blockDim.x) v_tile[idx] = e.v[(size_t)m0 * r + idx];
        __syncthreads();
      }
      for (int idx = tid; idx < RB * cnt; idx += blockDim.x) {
        const int t = idx / RB, row = idx - t * RB;
        const int nn = n0 + row;
        if (nn < N) {
          float yv = yacc[(m0 + t) * YS + row];
          const uint16_t* br = bpre ? bs + row * r : a.B + (size_t)nn * r;
          const float* vr = v_tile + t * r;
          for (int j = 0; j < r; ++j) yv += act2f<DT>(br[j]) * vr[j];
          a.y[(size_t)(m0 + t) * N + nn] = f2act<DT>(yv);
        }
      }
      __syncthreads();
    }
  }
  if constexpr (EPI == EPI_FUSED) fused_exit(a, gen);
}

// ---------------------------------------------------------------------------
// Prefill GEMM: 128x128 output tile per block (tokens x rows), K staged 64 at
// a time through double-buffered LDS; the packed codes are dequantised once
// per block into the LDS tile, (q - z) exact then times s with one rounding
// (fp16) or via fp32 (bf16). Four waves, 2x2, each 64x64 = 4x4 MFMA tiles.
// ---------------------------------------------------------------------------
template <int DT>
__device__ __forceinline__ void dequant_word_pairs(uint32_t w, float s, int z, uint32_t out[4]) {
  // natural order pairs (q0,q1), (q2,q3), (q4,q5), (q6,q7)
  const uint32_t lo = w & 0x0F0F0F0Fu;         // q0 q2 q4 q6
  const uint32_t hi = (w >> 4) & 0x0F0F0F0Fu;  // q1 q3 q5 q7
  uint32_t p[4];
  p[0] = __builtin_amdgcn_perm(hi, lo, 0x0C040C00u);
  p[1] = __builtin_amdgcn_perm(hi, lo, 0x0C050C01u);
  p[2] = __builtin_amdgcn_perm(hi, lo, 0x0C060C02u);
  p[3] = __builtin_amdgcn_perm(hi, lo, 0x0C070C03u);
  if constexpr (DT == DT_F16) {
    const _Float16 zb = (_Float16)(1024 + z);
    const f16x2 nz = f16x2{-zb, -zb};
    const f16x2 s2 = f16x2{(_Float16)s, (_Float16)s};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f16x2 q = __builtin_bit_cast(f16x2, p[i] | 0x64006400u);
      out[i] = __builtin_bit_cast(uint32_t, (q + nz) * s2);
    }
  } else {
    const float zf = (float)z;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float a0 = ((float)(p[i] & 0xFFFF) - zf) * s;
      const float a1 = ((float)(p[i] >> 16) - zf) * s;
      out[i] = (uint32_t)f2act<DT>(a0) | ((uint32_t)f2act<DT>(a1) << 16);
    }
  }
}

template <int DT, int EPI>
__global__ __launch_bounds__(256) void k_gemm(GemmParams a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int LR = kGemmLdsRow;
  constexpr int TILE = kGemmTM * LR;  // halves per LDS tile
  uint16_t* Xs = (uint16_t*)smem;             // [2][128][LR]
  uint16_t* Ws = Xs + 2 * TILE;               // [2][128][LR]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = a.M, N = a.N, K = a.K;
  const int tiles_n = (N + kGemmTN - 1) / kGemmTN;
  const int m0 = (blockIdx.x / tiles_n) * kGemmTM;
  const int n0 = (blockIdx.x % tiles_n) * kGemmTN;
  const int KT = K / kGemmTK;

  // per-thread global load assignments (bounds-checked buffer loads)
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)M * K * 2);
  const rsrc_t rq = make_rsrc(a.qw, (uint32_t)N * (K / 2));
  const rsrc_t rsc = make_rsrc(a.sc, (uint32_t)N * a.ngroups * 2);
  const rsrc_t rz = make_rsrc(a.zr, (uint32_t)N * a.ngroups);
  int xr[4], xc[4];
  uint32_t xoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    xr[i] = c >> 3;
    xc[i] = (c & 7) * 8;
    xoff[i] = m0 + xr[i] < M ? ((uint32_t)(m0 + xr[i]) * K + xc[i]) * 2 : kOOB;
  }
  const int wr = tid >> 1, wh = tid & 1;
  const int wn_row = n0 + wr;
  const bool wok = wn_row < N;
  const uint32_t woff = wok ? (uint32_t)wn_row * (K / 2) + 16 * wh : kOOB;

  u32x4 xreg[4];
  u32x4 wreg;
  float sreg;
  int zreg;
  auto gload = [&](int kt) {
    const uint32_t k0 = (uint32_t)kt * kGemmTK;
#pragma unroll
    for (int i = 0; i < 4; ++i) xreg[i] = bld128(rx, xoff[i] + k0 * 2);
    wreg = bld128(rq, woff + k0 / 2);
    const uint32_t g = k0 / a.G;
    sreg = h2f((uint16_t)bld16(rsc, wok ? ((uint32_t)wn_row * a.ngroups + g) * 2 : kOOB));
    zreg = (int)bld8(rz, wok ? (uint32_t)wn_row * a.ngroups + g : kOOB);
  };
  auto lstore = [&](int buf) {
    uint16_t* xs = Xs + buf * TILE;
    uint16_t* ws = Ws + buf * TILE;
#pragma unroll
    for (int i = 0; i < 4; ++i) *(u32x4*)(xs + xr[i] * LR + xc[i]) = xreg[i];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      uint32_t o[4];
      dequant_word_pairs<DT>(wreg[c], sreg, zreg, o);
      *(u32x4*)(ws + wr * LR + 32 * wh + 8 * c) = u32x4{o[0], o[1], o[2], o[3]};
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) gload(kt + 1);
    const uint16_t* xs = Xs + buf * TILE;
    const uint16_t* ws = Ws + buf * TILE;
#pragma unroll
    for (int kk = 0; kk < kGemmTK; kk += 32) {
      u32x4 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const u32x4*)(xs + (wm * 64 + 16 * i + lr) * LR + kk + 8 * lg);
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = *(const u32x4*)(ws + (wn * 64 + 16 * j + lr) * LR + kk + 8 * lg);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16<DT>(af[i], bf[j], acc[i][j]);
    }
    if (kt + 1 < KT) lstore(buf ^ 1);
    __syncthreads();
  }

  if constexpr (EPI == EPI_READY) {
    // y += v_hi B^T + v_lo B^T over the rank (zero-padded to vstride)
    const int r = a.r;
    const bool bvec = (r & 7) == 0;
    for (int kr = 0; kr < a.vstride; kr += 32) {
      const int kk = kr + 8 * lg;
      u32x4 vhf[4], vlf[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + wm * 64 + 16 * i + lr;
        const bool ok = m < M;
        vhf[i] = ok ? ldg16(a.vh + (size_t)m * a.vstride + kk) : u32x4{0, 0, 0, 0};
        vlf[i] = ok ? ldg16(a.vl + (size_t)m * a.vstride + kk) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + 16 * j + lr;
        u32x4 f = u32x4{0, 0, 0, 0};
        if (n < N) {
          const uint16_t* br = a.B + (size_t)n * r;
          if (bvec) {
            if (kk < r) f = ldg16(br + kk);
          } else {
            uint32_t h[8];
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2) h[e2] = (kk + e2 < r) ? br[kk + e2] : 0u;
            f = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
          }
        }
        bfr[j] = f;
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = mfma16<DT>(vhf[i], bfr[j], acc[i][j]);
          acc[i][j] = mfma16<DT>(vlf[i], bfr[j], acc[i][j]);
        }
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + wn * 64 + 16 * j + lr;
      if (n >= N) continue;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int m = m0 + wm * 64 + 16 * i + 4 * lg + e2;
        if (m < M) a.y[(size_t)m * N + n] = f2act<DT>(acc[i][j][e2]);
      }
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
// Raise a kernel's dynamic-LDS limit when a launch needs more than 64 KB.
template <typename F>
static hipError_t allow_lds(F* fn, size_t lds) {
  if (lds <= 65536) return hipSuccess;
  return hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

#define SPEAR_DT_SWITCH(dt, ...)          \
  do {                                    \
    if ((dt) == DT_F16) {                 \
      constexpr int DTC = DT_F16;         \
      __VA_ARGS__;                        \
    } else {                              \
      constexpr int DTC = DT_BF16;        \
      __VA_ARGS__;                        \
    }                                     \
  } while (0)

hipError_t launch_dequant(int dt, const uint32_t* qw, const uint16_t* sc, const uint8_t* zr,
                          uint16_t* out, int N, int K, int G, hipStream_t st) {
  const long long nwords = (long long)N * (K / 8);
  const unsigned grid = (unsigned)((nwords + 255) / 256);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, hipLaunchKernelGGL(k_dequant<DTC>, dim3(grid), dim3(256), 0, st, qw, sc, zr,
                                         out, N, K, G));
  return hipGetLastError();
}

hipError_t launch_ec(int dt, const EcParams& e, int ntb, int block, size_t lds, hipStream_t st) {
  const unsigned grid = (unsigned)(ntb * e.P);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, {
    hipError_t err = allow_lds(k_ec<DTC>, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_ec<DTC>, dim3(grid), dim3(block), lds, st, e);
  });
  return hipGetLastError();
}

hipError_t launch_gate(int dt, const EcParams& e, int ntb, size_t lds, hipStream_t st) {
  if (ntb == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, {
    hipError_t err = allow_lds(k_gate<DTC>, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_gate<DTC>, dim3(ntb), dim3(256), lds, st, e);
  });
  return hipGetLastError();
}

hipError_t launch_ec_up_acc(int dt, const float* v, const uint16_t* B, uint16_t* y, int M, int N,
                            int r, hipStream_t st) {
  const long long total = (long long)M * N;
  const unsigned grid = (unsigned)((total + 255) / 256);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, hipLaunchKernelGGL(k_ec_up_acc<DTC>, dim3(grid), dim3(256), 0, st, v, B, y,
                                         M, N, r));
  return hipGetLastError();
}

template <int DT, int MT, int RT>
static hipError_t gemv_launch(int epi, const GemvParams& p, int grid, int block, size_t lds,
                              hipStream_t st) {
  hipError_t err = epi == EPI_NONE    ? allow_lds(k_gemv<DT, MT, RT, EPI_NONE>, lds)
                   : epi == EPI_READY ? allow_lds(k_gemv<DT, MT, RT, EPI_READY>, lds)
                                      : allow_lds(k_gemv<DT, MT, RT, EPI_FUSED>, lds);
  if (err != hipSuccess) return err;
  if (epi == EPI_NONE)
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_NONE>), dim3(grid), dim3(block), lds, st, p);
  else if (epi == EPI_READY)
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_READY>), dim3(grid), dim3(block), lds, st, p);
  else
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_FUSED>), dim3(grid), dim3(block), lds, st, p);
  return hipGetLastError();
}

// The GEMV shapes compiled in: (token tiles MT, row tiles RT).
// gemv_shape_supported() mirrors this list for the planner.
#define SPEAR_GEMV_SHAPES(X) \
  X(1, 1) X(1, 2) X(1, 4) X(2, 1) X(2, 2) X(2, 4) X(3, 1) X(3, 2) X(4, 1)

bool gemv_shape_supported(int MT, int RT) {
#define SPEAR_GEMV_MATCH(mt, rt) if (MT == mt && RT == rt) return true;
  SPEAR_GEMV_SHAPES(SPEAR_GEMV_MATCH)
#undef SPEAR_GEMV_MATCH
  return false;
}

hipError_t launch_gemv(int dt, int MT, int RT, int epi, const GemvParams& p, int grid, int block,
                       size_t lds, hipStream_t st) {
  if (grid == 0) return hipSuccess;
#define SPEAR_GEMV_CASE(mt, rt)                                                     \
  if (MT == mt && RT == rt)                                                         \
    return dt == DT_F16 ? gemv_launch<DT_F16, mt, rt>(epi, p, grid, block, lds, st) \
                        : gemv_launch<DT_BF16, mt, rt>(epi, p, grid, block, lds, st);
  SPEAR_GEMV_SHAPES(SPEAR_GEMV_CASE)
#undef SPEAR_GEMV_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_gemm(int dt, int epi, const GemmParams& p, hipStream_t st) {
  const int tm = (p.M + kGemmTM - 1) / kGemmTM, tn = (p.N + kGemmTN - 1) / kGemmTN;
  const unsigned grid = (unsigned)(tm * tn);
  if (grid == 0) return hipSuccess;
  const size_t lds = (size_t)4 * kGemmTM * kGemmLdsRow * 2;
  SPEAR_DT_SWITCH(dt, {
    if (epi == EPI_NONE) {
      hipError_t err = allow_lds(k_gemm<DTC, EPI_NONE>, lds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL((k_gemm<DTC, EPI_NONE>), dim3(grid), dim3(256), lds, st, p);
    } else {
      hipError_t err = allow_lds(k_gemm<DTC, EPI_READY>, lds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL((k_gemm<DTC, EPI_READY>), dim3(grid), dim3(256), lds, st, p);
    }
  });
  return hipGetLastError();
}

}  // namespace spear
