// gfx950 (MI355X) kernels of the W4+EC linear layer.
//
// Y = X . What^T + alpha * (gate (.) (X . A^T)) . B^T      (SPEAR, section 3.1, Eq. 3)
// What[n][k] = (q[n][k] - z[n][k/G]) * s[n][k/G]          (sections 2.1, 5.1)
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

#include <type_traits>
#include <stdint.h>

#include "spear_internal.h"

// This translation unit's weight-code width: the kernels that read the
// packed codes are instantiated for SPEAR_WB (4 or 3) and their launchers
// carry it in their names (launch_gemv_w4, launch_gemv_w3, ...); the build
// compiles this file once per width. Kernels that do not read the codes are
// compiled with the 4-bit unit only.
#ifndef SPEAR_WB
#define SPEAR_WB 4
#endif
#define SPEAR_CAT2(a, b) a##b
#define SPEAR_CAT(a, b) SPEAR_CAT2(a, b)
#define SPEAR_W(name) SPEAR_CAT(name, SPEAR_CAT(_w, SPEAR_WB))

namespace spear {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));

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

// 32 x 32 x 16 MFMA: lane l holds A row l % 32 and B column l % 32, each at
// K 8 (l / 32) .. +8; result element i of lane l is D[8 (i / 4) + 4 (l / 32)
// + i % 4][l % 32]
typedef float f32x16 __attribute__((ext_vector_type(16)));
template <int DT>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (DT == DT_F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
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
// 3-bit codes: a block of 32 codes c_0..c_31 in three words (w[0], w[1]:
// two-bit low fields, c_{2i} in bits 2i..2i+1 and c_{2i+1} in bits
// 16+2i..17+2i of w[0] for i < 8, of w[1] for i >= 8; w[2]: the high bits,
// c_{2i} at bit i and c_{2i+1} at bit 16+i). Pair p = (c_{2p}, c_{2p+1}),
// in natural K order, as two 16-bit lanes; `kg` = 0 gives the codes
// themselves, the magic pair (above) the biased act-dtype values.
__device__ __forceinline__ uint32_t w3_pair(const u32x4& w, int p, uint32_t kg) {
  const uint32_t lo = p < 8 ? w[0] : w[1];
  const uint32_t l = (lo >> (2 * (p & 7))) & 0x00030003u;
  const uint32_t h = (p >= 2 ? (w[2] >> (p - 2)) : (w[2] << (2 - p))) & 0x00040004u;
  return l | h | kg;
}
// MFMA operand jj (codes 8 jj .. 8 jj + 7 of the block, natural order) as
// biased act-dtype values
__device__ __forceinline__ u32x4 unpack3_biased(const u32x4& w, int jj, uint32_t kg) {
  return u32x4{w3_pair(w, 4 * jj, kg), w3_pair(w, 4 * jj + 1, kg), w3_pair(w, 4 * jj + 2, kg),
               w3_pair(w, 4 * jj + 3, kg)};
}
// Bytes of one row of packed codes.
template <int WB>
__host__ __device__ __forceinline__ uint32_t row_code_bytes(int K) {
  return WB == 4 ? (uint32_t)K / 2 : (uint32_t)K / 8 * 3;
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

// INT8 per-channel symmetric codes (the EC factors' deployment format):
// code q of channel c stands for sa[c] * q. Where a code feeds an MFMA it is
// dequantised to the activation dtype like the 4-bit weights, one rounding
// of the fp32 product s * q (exact for |q| <= 127). Bytes 2p and 2p + 1 of w.
template <int DT>
__device__ __forceinline__ uint32_t i8pair_to_act(uint32_t w, int p, float s) {
  const int b0 = (int)(w << (24 - 16 * p)) >> 24;
  const int b1 = (int)(w << (16 - 16 * p)) >> 24;
  return (uint32_t)f2act<DT>((float)b0 * s) | ((uint32_t)f2act<DT>((float)b1 * s) << 16);
}
// eight codes (two dwords, K order) -> an 8-element MFMA operand
template <int DT>
__device__ __forceinline__ u32x4 i8x8_to_act(uint32_t w0, uint32_t w1, float s) {
  return u32x4{i8pair_to_act<DT>(w0, 0, s), i8pair_to_act<DT>(w0, 1, s),
               i8pair_to_act<DT>(w1, 0, s), i8pair_to_act<DT>(w1, 1, s)};
}
template <int DT>
__device__ __forceinline__ uint16_t i8_to_act(int8_t q, float s) {
  return f2act<DT>((float)q * s);
}
// Eight INT8 codes as exact activation-dtype integers (|q| <= 127 is exact
// in both), for kernels that apply the scale to the fp32 result instead.
// fp16: the byte q + 128 is placed under the exponent of 1024 (0x64 high
// byte gives 1024 + b exactly) and 1152 is subtracted; bf16: through fp32.
template <int DT>
__device__ __forceinline__ u32x4 i8x8_exact(uint32_t w0, uint32_t w1) {
  if constexpr (DT == DT_F16) {
    const uint32_t b0 = w0 ^ 0x80808080u, b1 = w1 ^ 0x80808080u;
    const f16x2 off = f16x2{(_Float16)-1152.f, (_Float16)-1152.f};
    auto pr = [&](uint32_t b, uint32_t sel) {
      return __builtin_bit_cast(uint32_t,
                                __builtin_bit_cast(f16x2, __builtin_amdgcn_perm(0x64646464u, b, sel)) + off);
    };
    return u32x4{pr(b0, 0x04010400u), pr(b0, 0x04030402u), pr(b1, 0x04010400u), pr(b1, 0x04030402u)};
  } else {
    auto pr = [&](uint32_t w, int p) {
      const float a0 = (float)((int)(w << (24 - 16 * p)) >> 24);
      const float a1 = (float)((int)(w << (16 - 16 * p)) >> 24);
      return (__float_as_uint(a0) >> 16) | (__float_as_uint(a1) & 0xFFFF0000u);
    };
    return u32x4{pr(w0, 0), pr(w0, 1), pr(w1, 0), pr(w1, 1)};
  }
}

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
// 16 bytes per lane from `r` at byte offset `off` straight into LDS: lane l
// of the wave writes lds + 16 l (lds wave-uniform, 1 KB per instruction);
// completion is counted by vmcnt
__device__ __forceinline__ void bld128_lds(rsrc_t r, void* lds, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0, 0);
}
// voffset (per lane, carries the mask) + soffset (wave-uniform)
__device__ __forceinline__ u32x4 bld128s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
// 12 bytes (one block of 3-bit codes) into the first three lanes of a u32x4
__device__ __forceinline__ u32x4 bld96s(rsrc_t r, uint32_t voff, uint32_t soff) {
  const u32x3 v = __builtin_amdgcn_raw_buffer_load_b96(r, voff, soff, 0);
  return u32x4{v[0], v[1], v[2], 0u};
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
// 16-byte agent-scope (sc1) buffer store and load
__device__ __forceinline__ void bst128c(rsrc_t r, uint32_t off, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, 0x10);
}
__device__ __forceinline__ f32x4 bld128cf(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0x10));
}
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
// Coherent reads of data other workgroups published in this launch: buffer
// loads with the sc1 bit (what a relaxed agent-scope atomic load is on
// gfx950), bounds-checked so that every load of a batch is issued without a
// branch. A thread's loads go out four at a time, all in flight together.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t bld32c(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0x10);
}
__device__ __forceinline__ u32x2 bld64(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}
__device__ __forceinline__ u32x2 bld64c(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0x10);
}

// dst[i] = fp32 word at byte offset off(i) of `r`, i in [0, n). (Four named
// registers rather than an array: the loads must stay out of scratch.)
template <class Off>
__device__ __forceinline__ void gather_f32(rsrc_t r, int n, Off off, float* dst) {
  const int nthr = blockDim.x;
  for (int i0 = threadIdx.x; i0 < n; i0 += 4 * nthr) {
    const int i1 = i0 + nthr, i2 = i1 + nthr, i3 = i2 + nthr;
    const uint32_t w0 = bld32c(r, off(i0));
    const uint32_t w1 = bld32c(r, i1 < n ? off(i1) : kOOB);
    const uint32_t w2 = bld32c(r, i2 < n ? off(i2) : kOOB);
    const uint32_t w3 = bld32c(r, i3 < n ? off(i3) : kOOB);
    dst[i0] = __uint_as_float(w0);
    if (i1 < n) dst[i1] = __uint_as_float(w1);
    if (i2 < n) dst[i2] = __uint_as_float(w2);
    if (i3 < n) dst[i3] = __uint_as_float(w3);
  }
}

// Same for tagged words (tag << 32 | fp32 bits); returns 1 if any word this
// thread read carries another tag.
template <class Off>
__device__ __forceinline__ int gather_tagged(rsrc_t r, int n, Off off, uint32_t tag, float* dst) {
  const int nthr = blockDim.x;
  int stale = 0;
  for (int i0 = threadIdx.x; i0 < n; i0 += 4 * nthr) {
    const int i1 = i0 + nthr, i2 = i1 + nthr, i3 = i2 + nthr;
    const u32x2 w0 = bld64c(r, off(i0));
    const u32x2 w1 = bld64c(r, i1 < n ? off(i1) : kOOB);
    const u32x2 w2 = bld64c(r, i2 < n ? off(i2) : kOOB);
    const u32x2 w3 = bld64c(r, i3 < n ? off(i3) : kOOB);
    stale |= w0[1] != tag;
    dst[i0] = __uint_as_float(w0[0]);
    if (i1 < n) { stale |= w1[1] != tag; dst[i1] = __uint_as_float(w1[0]); }
    if (i2 < n) { stale |= w2[1] != tag; dst[i2] = __uint_as_float(w2[0]); }
    if (i3 < n) { stale |= w3[1] != tag; dst[i3] = __uint_as_float(w3[0]); }
  }
  return stale;
}

// out(i, sum over q < P of the word at off(q, i)), i in [0, n), summed in
// slice order; the words go through `scratch` (cap floats of LDS) in chunks.
// Every thread of the block calls it; it ends with a barrier.
template <class Off, class Out>
__device__ void sum_slices(rsrc_t r, int P, int n, Off off, float* scratch, int cap, Out out) {
  const int C = max(1, cap / P);
  for (int e0 = 0; e0 < n; e0 += C) {
    const int c = min(C, n - e0);
    gather_f32(r, P * c, [&](int i) {
      const int q = i / c;
      return off(q, e0 + (i - q * c));
    }, scratch);
    __syncthreads();
    for (int i = threadIdx.x; i < c; i += blockDim.x) {
      float v = 0.f;
      for (int q = 0; q < P; ++q) v += scratch[q * c + i];
      out(e0 + i, v);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// EC projection of one token tile over iterations [it_beg, it_end) and row
// tiles [t_beg, t_end) of R = [A; w_g] (R1 rows; the gate row w_g is row r):
// u_lds[t][j] = sum_k x[16*tb + t][k] * R[j][k] for the rows of those tiles.
// Each wave takes IPP iterations per pass with all of their loads issued
// first; the waves' partial tiles are summed in LDS in a fixed order (wave 0
// first), so the result does not depend on timing.
// ---------------------------------------------------------------------------
template <int DT, int IPP>
__device__ void ec_project(const EcParams& e, int tb, int it_beg, int it_end, int t_beg, int t_end,
                           float* u_lds, float* red) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int NW = blockDim.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // token rows past M read row M-1: their results are never used
  const int m = min(tb * kTokTile + lr, e.M - 1);
  const rsrc_t rx = make_rsrc(e.x, (uint32_t)e.M * e.K * 2);
  const bool i8 = e.A8 != nullptr;  // uniform
  const rsrc_t ra = i8 ? make_rsrc(e.A8, (uint32_t)e.r * e.K) : make_rsrc(e.A, (uint32_t)e.r * e.K * 2);
  const rsrc_t rg = make_rsrc(e.wg, e.gate == GATE_SIGMOID ? (uint32_t)e.K * 2 : 0u);
  // K order within an iteration: MFMA jj, lane group lg takes K
  // [8 lg + 32 jj, +8) for both operands, so that each load reads 64
  // contiguous bytes per row (the MFMA lane layout would otherwise spread a
  // load over twice as many cache lines)
  const uint32_t xoff = (uint32_t)m * e.K * 2 + 16 * lg;
  for (int tg0 = t_beg; tg0 < t_end; tg0 += kEcTiles) {
    const int nt = min(kEcTiles, t_end - tg0);
    f32x4 acc[kEcTiles];
    uint32_t aoff[kEcTiles], goff[kEcTiles];
    bool has_g[kEcTiles];
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t) {
      acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int j = (tg0 + t) * 16 + lr;
      aoff[t] = (t < nt && j < e.r) ? (uint32_t)j * e.K * 2 + 16 * lg : kOOB;
      goff[t] = (t < nt && j == e.r && e.gate == GATE_SIGMOID) ? 16u * lg : kOOB;
      // uniform: does this row tile hold the gate row?
      has_g[t] = t < nt && e.gate == GATE_SIGMOID && e.r >= (tg0 + t) * 16 &&
                 e.r < (tg0 + t + 1) * 16;
    }
    // the gate row's tile (uniform), or -1; w_g goes to registers of its own
    // and joins that tile's operand only at the MFMA (a value combined right
    // after its load would make the wave wait for every earlier load)
    int gt = -1;
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t)
      if (has_g[t]) gt = t;
    uint32_t goff_g = kOOB;
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t)
      if (t == gt) goff_g = goff[t];
    // the iterations, for act-dtype A (16-byte loads) or INT8 A (8-byte
    // loads of the same eight K, dequantised with the row's scale at the MFMA)
    auto iterate = [&](auto i8c) {
      constexpr bool kI8 = decltype(i8c)::value;
      float sa[kEcTiles];
#pragma unroll
      for (int t = 0; t < kEcTiles; ++t) {
        const int j = (tg0 + t) * 16 + lr;
        sa[t] = kI8 && t < nt && j < e.r ? e.sa[j] : 0.f;
      }
      for (int it0 = it_beg + wave * IPP; it0 < it_end; it0 += NW * IPP) {
        u32x4 xv[IPP][4], av[IPP][kEcTiles][4], gv[IPP][4];
#pragma unroll
        for (int h = 0; h < IPP; ++h) {
          const bool ok = it0 + h < it_end;  // uniform
          const uint32_t kb = (uint32_t)(it0 + h) * (kIterK * 2);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) xv[h][jj] = bld128(rx, ok ? xoff + kb + 64 * jj : kOOB);
#pragma unroll
          for (int t = 0; t < kEcTiles; ++t)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              if constexpr (kI8) {
                // aoff[t] and kb count 2-byte elements twice: halve them
                const u32x2 q = bld64(ra, ok && aoff[t] != kOOB ? (aoff[t] + kb) / 2 + 32 * jj : kOOB);
                av[h][t][jj] = u32x4{q[0], q[1], 0u, 0u};
              } else {
                av[h][t][jj] = bld128(ra, ok && aoff[t] != kOOB ? aoff[t] + kb + 64 * jj : kOOB);
              }
            }
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            gv[h][jj] = bld128(rg, ok && goff_g != kOOB ? goff_g + kb + 64 * jj : kOOB);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int h = 0; h < IPP; ++h)
#pragma unroll
          for (int t = 0; t < kEcTiles; ++t)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              u32x4 af = av[h][t][jj];
              if constexpr (kI8) af = i8x8_to_act<DT>(af[0], af[1], sa[t]);
              acc[t] = mfma16<DT>(t == gt ? (af | gv[h][jj]) : af, xv[h][jj], acc[t]);
            }
      }
    };
    if (i8) iterate(std::true_type{});
    else iterate(std::false_type{});
    // lane l holds token l % 16 and rows 4 * (l / 16) .. + 3 of each tile
#pragma unroll
    for (int t = 0; t < kEcTiles; ++t)
      *(f32x4*)(red + ((wave * kEcTiles + t) * 64 + lane) * 4) = acc[t];
    __syncthreads();
    for (int idx = tid; idx < nt * 256; idx += blockDim.x) {
      const int t = idx >> 8, rem = idx & 255, ln = rem >> 2, i = rem & 3;
      float s = 0.f;
      for (int w = 0; w < NW; ++w) s += red[((w * kEcTiles + t) * 64 + ln) * 4 + i];
      const int j = (tg0 + t) * 16 + 4 * (ln >> 4) + i;
      if (j < e.R1) u_lds[(ln & 15) * e.R1p + j] = s;
    }
    __syncthreads();
  }
}

// The paper's rank-space gate for cnt tokens at once, by the whole block:
// hid = ReLU(W1 u + b1) for every token, then v = alpha (1 + tanh(W2 hid +
// b2)) (.) u, in fp32, cap tokens per pass (hid holds cap x h floats). u
// rows are us floats apart, v rows vs. With wst (LDS room for
// tanh_stage_halves(h, r) halves, or null) the gate's parameters are first
// copied there with coalesced loads, so that the dot products read LDS
// rather than one global load per term. Ends with a barrier.
template <int DT>
__device__ void tanh_gate_tokens(int cnt, int r, int h, const float* u, int us,
                                 const uint16_t* W1, const uint16_t* b1, const uint16_t* W2,
                                 const uint16_t* b2, float alpha, float* hid, int cap, float* v,
                                 int vs, uint16_t* wst) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  if (wst) {
    const int n1 = h * r, n2 = n1 + h, n3 = n2 + r * h, n4 = n3 + r;
    for (int i = tid; i < n4; i += nthr)
      wst[i] = i < n1 ? W1[i] : i < n2 ? b1[i - n1] : i < n3 ? W2[i - n2] : b2[i - n3];
    __syncthreads();
    W1 = wst;
    b1 = wst + n1;
    W2 = wst + n2;
    b2 = wst + n3;
  }
  for (int t0 = 0; t0 < cnt; t0 += cap) {
    const int c = min(cap, cnt - t0);
    for (int idx = tid; idx < c * h; idx += nthr) {
      const int t = idx / h, i = idx - t * h;
      const float* ut = u + (t0 + t) * us;
      const uint16_t* w1 = W1 + (size_t)i * r;
      float a = act2f<DT>(b1[i]);
      for (int j = 0; j < r; ++j) a += act2f<DT>(w1[j]) * ut[j];
      hid[idx] = a > 0.f ? a : 0.f;
    }
    __syncthreads();
    for (int idx = tid; idx < c * r; idx += nthr) {
      const int t = idx / r, j = idx - t * r;
      const float* ht = hid + t * h;
      const uint16_t* w2 = W2 + (size_t)j * h;
      float a = act2f<DT>(b2[j]);
      for (int i = 0; i < h; ++i) a += act2f<DT>(w2[i]) * ht[i];
      v[(t0 + t) * vs + j] = alpha * (1.f + tanhf(a)) * u[(t0 + t) * us + j];
    }
    __syncthreads();
  }
}

// Gate of one token tile: from u (LDS, [16][R1p]) to v_tile (LDS, [16][r]):
// v = alpha * g * u (sigmoid-linear), alpha * (1 + tanh(W2 ReLU(W1 u + b1) + b2)) (.) u
// (tanh-MLP), or alpha * u (gate one). Ends with a barrier.
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

// One EC producer workgroup b: token tile, K-slice and row-tile group from b.
// It projects its share; then (EC_GATHER) publishes its tagged partial sums
// for the consumers to add up, or joins the last-arriver reduction of its
// token tile, whose last workgroup sums the slices in order, applies the gate
// and publishes v: as fp32 (read by a later kernel), as act-dtype hi/lo parts
// (the prefill GEMM epilogue) and/or as tagged words in one copy per XCD (the
// fused kernel's consumers).
template <int DT, int IPP>
__device__ __forceinline__ void ec_producer(const EcParams& e, int b, uint32_t gen, char* smem) {
  __shared__ int s_last;
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int NW = nthr >> 6;
  const int IT = e.K / kIterK;
  const int per_tb = e.P * e.PG;
  const int tb = b / per_tb, rem = b - tb * per_tb;
  const int pk = rem / e.PG, pg = rem - pk * e.PG;
  const int it_beg = pk * e.ips, it_end = min(IT, it_beg + e.ips);
  const int RTe = (e.R1 + 15) >> 4;
  const int t_beg = pg * e.tpg, t_end = min(RTe, t_beg + e.tpg);
  float* red = (float*)smem;
  char* es = smem + ec_red_bytes(NW);
  float* u_lds = (float*)(es + ec_lds_u_off());
  float* hid = (float*)(es + ec_lds_hid_off(e.R1p));
  float* v_tile = (float*)(es + ec_lds_v_off(e.R1p, e.h));
  const int m0 = tb * kTokTile;
  const int cnt = min(kTokTile, e.M - m0);
  const int j_beg = 16 * t_beg, nj = min(e.R1, 16 * t_end) - j_beg;

  ec_project<DT, IPP>(e, tb, it_beg, it_end, t_beg, t_end, u_lds, red);

  if (e.mode == EC_GATHER) {
    const uint32_t tag = ec_tag(gen);
    const size_t per_copy = (size_t)e.P * e.M * e.R1;
    for (int idx = tid; idx < kVCopies * cnt * nj; idx += nthr) {
      const int c = idx / (cnt * nj), o = idx - c * (cnt * nj);
      const int t = o / nj, j = j_beg + (o - t * nj);
      const unsigned long long w =
          ((unsigned long long)tag << 32) | __float_as_uint(u_lds[t * e.R1p + j]);
      __hip_atomic_store(e.vtag + c * per_copy + ((size_t)pk * e.M + m0 + t) * e.R1 + j, w,
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // the data is complete before the ready counters count it
    complete_and_sync();
    if (tid < kVCopies)
      __hip_atomic_fetch_add(e.ready + tid * (kReadyStride / 8), (unsigned long long)publisher_increment(b, e.npub),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }

  if (per_tb > 1) {
    float* part = e.upart + ((size_t)tb * e.P + pk) * kTokTile * e.R1;
    for (int idx = tid; idx < cnt * nj; idx += nthr) {
      const int t = idx / nj, j = j_beg + (idx - t * nj);
      st_agent(part + t * e.R1 + j, u_lds[t * e.R1p + j]);
    }
    complete_and_sync();
    if (tid == 0) s_last = arrive_last(e.ctr + tb, (uint32_t)per_tb) ? 1 : 0;
    __syncthreads();
    if (!s_last) return;
    // the slices' partial tiles [P][cnt][R1], summed in slice order through
    // the wave-partials region (free now)
    const rsrc_t rp = make_rsrc(e.upart + (size_t)tb * e.P * kTokTile * e.R1,
                                (uint32_t)e.P * kTokTile * e.R1 * 4);
    sum_slices(rp, e.P, cnt * e.R1,
               [&](int q, int i) { return (uint32_t)(q * kTokTile * e.R1 + i) * 4u; }, red,
               (int)(ec_red_bytes(NW) / 4), [&](int i, float v) {
                 const int t = i / e.R1, j = i - t * e.R1;
                 u_lds[t * e.R1p + j] = v;
               });
  }

  if (e.mode == EC_RAW) {
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
      const float val = j < e.r ? v_tile[t * e.r + j] : 0.f;
      const uint16_t hi = f2act<DT>(val);
      const uint16_t lo = f2act<DT>(val - act2f<DT>(hi));
      e.vh[(size_t)(m0 + t) * e.vstride + j] = hi;
      e.vl[(size_t)(m0 + t) * e.vstride + j] = lo;
    }
  }
  if (e.vtag) {
    const uint32_t tag = ec_tag(gen);
    const size_t per_copy = (size_t)e.M * e.r;
    for (int idx = tid; idx < cnt * e.r * kVCopies; idx += nthr) {
      const int c = idx / (cnt * e.r), o = idx - c * (cnt * e.r);
      const unsigned long long w =
          ((unsigned long long)tag << 32) | __float_as_uint(v_tile[o]);
      __hip_atomic_store(e.vtag + c * per_copy + (size_t)m0 * e.r + o, w, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    complete_and_sync();
    if (tid < kVCopies)
      __hip_atomic_fetch_add(e.ready + tid * (kReadyStride / 8), (unsigned long long)publisher_increment(tb, e.npub),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// EC pre-kernel (semi-fused and chain paths): one producer per workgroup.
template <int DT, int IPP>
__global__ __launch_bounds__(512) void k_ec(EcParams e) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  ec_producer<DT, IPP>(e, blockIdx.x, 0u, smem);
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

// Naive chain, reprojection + accumulate: y[m][n] += sum_j v[m][j] B[n][j]
// (INT8 B: sb[n] * sum_j v[m][j] q[n][j], in fp32).
template <int DT>
__global__ __launch_bounds__(256) void k_ec_up_acc(const float* __restrict__ v,
                                                   const uint16_t* __restrict__ B,
                                                   const int8_t* __restrict__ B8,
                                                   const float* __restrict__ sb,
                                                   uint16_t* __restrict__ y, int M, int N, int r) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)M * N) return;
  const int m = (int)(idx / N), n = (int)(idx % N);
  float a = act2f<DT>(y[idx]);
  if (B8) {
    float t = 0.f;
    for (int j = 0; j < r; ++j) t += v[(size_t)m * r + j] * (float)B8[(size_t)n * r + j];
    a += sb[n] * t;
  } else {
    for (int j = 0; j < r; ++j) a += v[(size_t)m * r + j] * act2f<DT>(B[(size_t)n * r + j]);
  }
  y[idx] = f2act<DT>(a);
}

// Post-EC tail, next-layer RMSNorm: y_norm[m][n] = y[m][n] * rsqrt(mean_n y[m][n]^2
// + eps) * w[n] over the stored (rounded) row, in fp32, one rounding. One
// workgroup of 256 threads per token row; the sum of squares is reduced in a
// fixed order (per-thread strided sums, then a tree in LDS).
template <int DT>
__global__ __launch_bounds__(256) void k_rmsnorm(const uint16_t* __restrict__ y,
                                                 const uint16_t* __restrict__ w, float eps,
                                                 uint16_t* __restrict__ y_norm, int N) {
  __shared__ float red[256];
  const int m = blockIdx.x, tid = threadIdx.x;
  const uint16_t* yr = y + (size_t)m * N;
  float ss = 0.f;
  for (int n = tid; n < N; n += 256) {
    const float v = act2f<DT>(yr[n]);
    ss += v * v;
  }
  red[tid] = ss;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if (tid < h) red[tid] += red[tid + h];
    __syncthreads();
  }
  const float scale = 1.f / sqrtf(red[0] / (float)N + eps);
  uint16_t* out = y_norm + (size_t)m * N;
  for (int n = tid; n < N; n += 256) out[n] = f2act<DT>(act2f<DT>(yr[n]) * scale * act2f<DT>(w[n]));
}

// Every workgroup of the fused grid advances its class's launch counter once
// as it ends (see gen_increment): relaxed adds that nothing waits for.
__device__ __forceinline__ unsigned long long* gen_counter(const GemvParams& a, int block) {
  return a.ec.gen + (size_t)(block % kGenClasses) * (kGenStride / 8);
}
__device__ __forceinline__ void fused_exit(const GemvParams& a) {
  const int b = blockIdx.x;
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(gen_counter(a, b), (unsigned long long)gen_increment(b, a.grid_total),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // classes without a member in a small grid advance with workgroup 0
  if (b == 0 && (int)threadIdx.x >= a.grid_total && (int)threadIdx.x < kGenClasses)
    __hip_atomic_fetch_add(gen_counter(a, threadIdx.x), 1ull << 32, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// The GEMV's EC wave. In the EC variants every workgroup carries one wave
// beyond its GEMV waves; on the first K-slice it obtains v for each token
// tile and computes v B^T for the workgroup's rows while the GEMV waves
// stream the codes, so its waits (for the producers, for cold caches) stay
// off the critical path. Everything below is single-wave: lanes exchange data
// through LDS in program order, with no workgroup barrier.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void wave_sync() { __builtin_amdgcn_wave_barrier(); }

// dst[i] = fp32 part of the tagged word at off(i), i in [0, n), over the
// wave's 64 lanes; returns 1 (in every lane) if any word carries another tag.
// COH: coherent (sc1) loads, else loads through this XCD's L2, which are
// cheaper but may return a line cached before the data was published (its
// tag then tells). Nine loads per lane go out together (576 words), so that
// the EC data of a token tile at rank 64 (520 words in eight partials) costs
// one round trip, not three; more would push the fused GEMV past its
// 128-VGPR budget into scratch.
template <bool COH, class Off>
__device__ __forceinline__ bool gather_tagged_w(rsrc_t r, int n, Off off, uint32_t tag, float* dst) {
  const int lane = threadIdx.x & 63;
  constexpr int aux = COH ? 0x10 : 0;
  constexpr int U = 9;
  int stale = 0;
  for (int i0 = lane; i0 < n; i0 += 64 * U) {
    u32x2 w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + 64 * u;
      w[u] = __builtin_amdgcn_raw_buffer_load_b64(r, i < n ? off(i) : kOOB, 0, aux);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + 64 * u;
      if (i < n) {
        stale |= w[u][1] != tag;
        dst[i] = __uint_as_float(w[u][0]);
      }
    }
  }
  wave_sync();
  return __any(stale);
}

// u_lds[t][j] = sum_k x[16 tb + t][k] R[j][k] for all R1 rows and all of K,
// by one wave (the EC wave's fallback when the producers' data never came).
template <int DT>
__device__ void ec_project_wave(const EcParams& e, int tb, float* u_lds) {
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int IT = e.K / kIterK, RTe = (e.R1 + 15) >> 4;
  const int m = min(tb * kTokTile + lr, e.M - 1);
  const rsrc_t rx = make_rsrc(e.x, (uint32_t)e.M * e.K * 2);
  const bool i8 = e.A8 != nullptr;  // uniform
  const rsrc_t ra = i8 ? make_rsrc(e.A8, (uint32_t)e.r * e.K) : make_rsrc(e.A, (uint32_t)e.r * e.K * 2);
  const rsrc_t rg = make_rsrc(e.wg, e.gate == GATE_SIGMOID ? (uint32_t)e.K * 2 : 0u);
  // K order within an iteration: MFMA jj, lane group lg takes K
  // [8 lg + 32 jj, +8), so that each load reads 64 contiguous bytes per row
  const uint32_t xoff = (uint32_t)m * e.K * 2 + 16 * lg;
  for (int t = 0; t < RTe; ++t) {
    const int j = t * 16 + lr;
    const uint32_t aoff = j < e.r ? (uint32_t)j * e.K * 2 + 16 * lg : kOOB;
    const uint32_t goff = (j == e.r && e.gate == GATE_SIGMOID) ? 16u * lg : kOOB;
    const float saj = i8 && j < e.r ? e.sa[j] : 0.f;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < IT; ++it) {
      const uint32_t kb = (uint32_t)it * (kIterK * 2);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const u32x4 xv = bld128(rx, xoff + kb + 64 * jj);
        u32x4 av;
        if (i8) {
          const u32x2 q = bld64(ra, aoff != kOOB ? (aoff + kb) / 2 + 32 * jj : kOOB);
          av = i8x8_to_act<DT>(q[0], q[1], saj);
        } else {
          av = bld128(ra, aoff != kOOB ? aoff + kb + 64 * jj : kOOB);
        }
        av |= bld128(rg, goff != kOOB ? goff + kb + 64 * jj : kOOB);
        acc = mfma16<DT>(av, xv, acc);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int jr = t * 16 + 4 * lg + i;
      if (jr < e.R1) u_lds[lr * e.R1p + jr] = acc[i];
    }
  }
  wave_sync();
}

// The gate of one token tile by one wave: u_lds [16][R1p] -> v_tile [16][r].
template <int DT>
__device__ void ec_gate_wave(const EcParams& e, int cnt, const float* u_lds, float* hid,
                             float* v_tile) {
  const int lane = threadIdx.x & 63;
  const int r = e.r;
  if (e.gate == GATE_TANH) {
    for (int t = 0; t < cnt; ++t) {
      const float* u = u_lds + t * e.R1p;
      for (int i = lane; i < e.h; i += 64) {
        float a = act2f<DT>(e.b1[i]);
        const uint16_t* w1 = e.W1 + (size_t)i * r;
        for (int j = 0; j < r; ++j) a += act2f<DT>(w1[j]) * u[j];
        hid[i] = a > 0.f ? a : 0.f;
      }
      wave_sync();
      for (int j = lane; j < r; j += 64) {
        float a = act2f<DT>(e.b2[j]);
        const uint16_t* w2 = e.W2 + (size_t)j * e.h;
        for (int i = 0; i < e.h; ++i) a += act2f<DT>(w2[i]) * hid[i];
        v_tile[t * r + j] = e.alpha * (1.f + tanhf(a)) * u[j];
      }
      wave_sync();
    }
  } else {
    for (int idx = lane; idx < cnt * r; idx += 64) {
      const int t = idx / r, j = idx - t * r;
      float g = 1.f;
      if (e.gate == GATE_SIGMOID) {
        const float z = u_lds[t * e.R1p + r] + e.b_g;
        g = z >= 0.f ? 1.f / (1.f + __expf(-z)) : __expf(z) / (1.f + __expf(z));
      }
      v_tile[idx] = e.alpha * g * u_lds[t * e.R1p + j];
    }
    wave_sync();
  }
}

// The EC wave's work for the workgroup's rows n0 .. n0 + 16 RT: for every
// token tile, v (from the previous kernel, or from this grid's producers once
// their ready flags carry this launch's tag, or computed here on time-out),
// then ev = v B^T as two MFMAs per 32 ranks (v split into act-dtype high and
// low parts), stored per (row tile, token tile) in the layout of a GEMV
// wave's accumulators.
template <int DT, int MT, int RT, int EPI>
__device__ void ec_wave(const GemvParams& a, uint32_t gen, char* smem, int n0, bool bpre) {
  const EcParams& e = a.ec;
  const int lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const int M = a.M, N = a.N, r = a.r;
  char* es = smem + a.lds_e;
  float* u_lds = (float*)(es + ec_lds_u_off());
  float* hid = (float*)(es + ec_lds_hid_off(e.R1p));
  float* v_tile = (float*)(es + ec_lds_v_off(e.R1p, e.h));
  const uint16_t* bs = (const uint16_t*)(smem + a.lds_b);
  float* gsc = (float*)(smem + a.lds_g);
  float* evs = (float*)(smem + a.lds_ev);
  const rsrc_t rb = make_rsrc(a.B, (uint32_t)N * r * 2);
  const uint32_t tag = ec_tag(gen);
  const int copy = blockIdx.x % kVCopies;
  const int nkk = (r + 31) / 32;
  // ev = v B^T for token tile mt from v_tile, into the result tiles
  auto up_project = [&](int mt, int cnt) {
    f32x4 ev[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) ev[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kk = 0; kk < nkk; ++kk) {
      const int j0 = 32 * kk + 8 * lg;
      u32x4 ah, al;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = j0 + 2 * q;
        const float f0 = (lr < cnt && j < r) ? v_tile[lr * r + j] : 0.f;
        const float f1 = (lr < cnt && j + 1 < r) ? v_tile[lr * r + j + 1] : 0.f;
        const uint32_t h0 = f2act<DT>(f0), h1 = f2act<DT>(f1);
        ah[q] = h0 | (h1 << 16);
        al[q] = (uint32_t)f2act<DT>(f0 - act2f<DT>(h0)) |
                ((uint32_t)f2act<DT>(f1 - act2f<DT>(h1)) << 16);
      }
#pragma unroll
      for (int t = 0; t < RT; ++t) {
        const int row = 16 * t + lr, n = n0 + row;
        u32x4 bf;
        if (bpre && (r & 7) == 0 && j0 < r) {
          bf = *(const u32x4*)(bs + row * r + j0);
        } else {
          auto bval = [&](int j) -> uint32_t {
            if (n >= N || j >= r) return 0u;
            if (a.B8) return i8_to_act<DT>(a.B8[(size_t)n * r + j], a.sb[n]);
            return bpre ? (uint32_t)bs[row * r + j] : bld16(rb, (uint32_t)(n * r + j) * 2);
          };
#pragma unroll
          for (int q = 0; q < 4; ++q) bf[q] = bval(j0 + 2 * q) | (bval(j0 + 2 * q + 1) << 16);
        }
        ev[t] = mfma16<DT>(ah, bf, ev[t]);
        ev[t] = mfma16<DT>(al, bf, ev[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < RT; ++t) *(f32x4*)(evs + ((t * MT + mt) * 64 + lane) * 4) = ev[t];
    wave_sync();
  };

  if constexpr (EPI == EPI_READY) {
    for (int mt = 0; mt < MT; ++mt) {
      const int m0 = 16 * mt, cnt = min(16, M - m0);
      for (int idx = lane; idx < cnt * r; idx += 64) v_tile[idx] = e.v[(size_t)m0 * r + idx];
      wave_sync();
      up_project(mt, cnt);
    }
    return;
  }

  // Fused: one attempt reads the published data of token tile mt (tagged
  // words), completes v and its product, and tells whether every word was
  // current; a stale attempt still runs the whole path, which warms this
  // wave's caches while the producers finish. `dry` reads nothing.
  auto attempt = [&](int mt, int cnt, bool coh, bool dry) -> bool {
    const int m0 = 16 * mt;
    bool stale;
    if (e.mode == EC_GATHER) {
      const int per = cnt * e.R1;
      const size_t per_copy = (size_t)e.P * e.M * e.R1;
      const rsrc_t rv = make_rsrc(e.vtag + copy * per_copy, (uint32_t)(per_copy * 8));
      auto off = [&](int i) {
        const int q = i / per, o = i - q * per;
        return (uint32_t)(((size_t)q * e.M + m0) * e.R1 + o) * 8u;
      };
      const int n = dry ? 0 : e.P * per;
      stale = dry || (coh ? gather_tagged_w<true>(rv, n, off, tag, gsc)
                          : gather_tagged_w<false>(rv, n, off, tag, gsc));
      for (int idx = lane; idx < per; idx += 64) {
        float sum = 0.f;
        for (int q = 0; q < e.P; ++q) sum += gsc[q * per + idx];
        const int t = idx / e.R1, j = idx - t * e.R1;
        u_lds[t * e.R1p + j] = sum;
      }
      wave_sync();
      ec_gate_wave<DT>(e, cnt, u_lds, hid, v_tile);
    } else {
      const size_t per_copy = (size_t)e.M * r;
      const rsrc_t rv = make_rsrc(e.vtag + copy * per_copy, (uint32_t)(per_copy * 8));
      auto off = [&](int i) { return (uint32_t)((size_t)m0 * r + i) * 8u; };
      const int n = dry ? 0 : cnt * r;
      stale = dry || (coh ? gather_tagged_w<true>(rv, n, off, tag, v_tile)
                          : gather_tagged_w<false>(rv, n, off, tag, v_tile));
    }
    up_project(mt, cnt);
    return !stale;
  };

  // warm-up pass, then wait: small problems poll the tagged data itself;
  // the others wait (bounded) for this copy's ready counter to show every
  // publisher of this launch and then read the data once through the L2,
  // re-reading it coherently if a cached line was stale. (Coherent reads
  // from every EC wave at once were measured: hundreds of waves reading the
  // same few lines at the memory side delay the producers' own stores, 70B
  // q 44.7 us against 18.7 us.)
  bool ok = true;
  if (!e.direct) {
    attempt(0, min(16, M), false, true);
    const unsigned long long* rc = e.ready + copy * (kReadyStride / 8);
    const rsrc_t rr = make_rsrc(rc, 8);
    const unsigned long long goal = ((unsigned long long)gen + 1ull) << 32;
    for (int poll = 0;; ++poll) {
      const u32x2 c = bld64c(rr, 0u);
      const unsigned long long cv = ((unsigned long long)c[1] << 32) | c[0];
      // counts of this launch lie in [goal - 2^32, goal]; the difference is
      // taken modulo 2^64 so that wrap-around is harmless
      if ((long long)(cv - goal) >= 0) break;
      if (poll >= a.wait_polls) { ok = false; break; }
      __builtin_amdgcn_s_sleep(16);
    }
  }
  for (int mt = 0; mt < MT; ++mt) {
    const int cnt = min(16, M - 16 * mt);
    bool have = false;
    if (e.direct) {
      for (int k = 0; k <= a.wait_polls && !have; ++k) {
        have = attempt(mt, cnt, true, false);
        if (!have) __builtin_amdgcn_s_sleep(4);
      }
    } else if (ok) {
      have = attempt(mt, cnt, false, false) || attempt(mt, cnt, true, false);
    }
    if (!have) {
      ec_project_wave<DT>(e, mt, u_lds);
      ec_gate_wave<DT>(e, cnt, u_lds, hid, v_tile);
      up_project(mt, cnt);
    }
  }
}

// ---------------------------------------------------------------------------
// Decode GEMV. A block owns RT row tiles (16 rows each) and a K-slice of
// iterations (128 K each); each of its NW waves walks a contiguous chunk of
// that slice as a software pipeline: the codes of iteration it+1 are in
// flight while iteration it is computed. The block's slice of x is staged in
// LDS once when it fits (else read through the cache per iteration), and so
// are the scales and zero points of its rows. The MFMA multiplies
// activations (A operand, 16 token rows) by the biased codes (B operand, 16
// weight rows as columns), so each lane owns one weight row per tile and
// needs one scale and one zero point per iteration:
//   sum_k x (q - z) s = s * ( sum_k x (bias + q) - (bias + z) * sum_k x ),
// with sum_k x from an MFMA against ones, shared by the RT tiles.
// In the EC variants the block has one more wave, the EC wave (above), whose
// v B^T tiles join the waves' partial tiles in the fixed-order reduction of
// the first K-slice. K-slices are reduced through partial sums and a last
// arriver.
//
// Fused variant: the first n_prod blocks of the grid are EC producers; the
// others' EC waves wait for what they publish.
// ---------------------------------------------------------------------------
template <int DT, int MT, int RT, int EPI, int WB, int NST = 2>
__device__ __forceinline__ void gemv_body(const GemvParams& a, int bid, uint32_t gen, char* smem) {
  __shared__ int s_flag;
  constexpr bool kEC = EPI == EPI_READY || EPI == EPI_FUSED;  // with an EC wave
  constexpr bool kLoc = EPI == EPI_LOCAL || EPI == EPI_LOCAL_I8;
  constexpr bool kI8 = EPI == EPI_LOCAL_I8;  // INT8 A and B
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int NW = (blockDim.x >> 6) - (kEC ? 1 : 0);           // GEMV waves
  const bool gw = wave < NW;
  const int lr = lane & 15, lg = lane >> 4;
  constexpr int RB = 16 * RT;
  const int M = a.M, N = a.N, K = a.K, G = a.G;
  const int IT = K / kIterK;
  const int rg = bid / a.S, s = bid - (bid / a.S) * a.S;
  const int n0 = rg * RB;
  const int it_blk = s * a.ips;
  const int it_end = min(IT, it_blk + a.ips);
  const int iw_beg = gw ? it_blk + wave * a.iw : 0;
  const int iw_end = gw ? min(it_end, iw_beg + a.iw) : 0;
  const int r = a.r;

  const rsrc_t rq = make_rsrc(a.qw, (uint32_t)N * row_code_bytes<WB>(K));
  const rsrc_t rsc = make_rsrc(a.sc, (uint32_t)N * a.ngroups * 2);
  const rsrc_t rz = make_rsrc(a.zr, (uint32_t)N * a.ngroups);
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)M * K * 2);
  const rsrc_t rb = kI8 ? make_rsrc(a.B8, (uint32_t)N * r) : make_rsrc(a.B, (uint32_t)N * r * 2);

  // The residual of the post-EC tail: when the block's outputs are at most
  // one per thread (decode), each thread's element is fetched here with the
  // other prologue loads instead of right before its store. The load is
  // issued unconditionally (out of range, it reads nothing): a branch around
  // it would make the wait before the first compute cover every prologue load.
  const bool res_pre = a.res != nullptr && RB * M <= (int)blockDim.x;
  uint32_t resv;
  {
    const int m = tid / RB, row = tid - (tid / RB) * RB;
    const rsrc_t rres = make_rsrc(a.res, a.res ? (uint32_t)M * N * 2 : 0u);
    resv = bld16(rres, res_pre && tid < RB * M && n0 + row < N
                           ? ((uint32_t)m * N + n0 + row) * 2 : kOOB);
  }
  // the rows of B ([RB][r], contiguous) of the block that adds v B^T (the
  // first K-slice's with an EC wave; any slice's in EPI_LOCAL, whose last
  // arriver adds it) are fetched up front into LDS when two 16-byte chunks
  // per thread cover them
  // (INT8 B: the codes, 16 per chunk, and then the rows' fp32 scales)
  constexpr int BCH = 2;
  const bool bpre = ((kEC && s == 0) || kLoc) && a.bpre;
  const int bchunks = kI8 ? RB * r / 16 : RB * r / 8;
  u32x4 bst[BCH];
  uint32_t sbst = 0;
  if (bpre) {
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int ci = tid + c * (int)blockDim.x;
      bst[c] = bld128(rb, ci < bchunks ? (uint32_t)n0 * r * (kI8 ? 1 : 2) + 16u * ci : kOOB);
    }
    if constexpr (kI8) {
      const rsrc_t rsb = make_rsrc(a.sb, (uint32_t)N * 4);
      sbst = __builtin_amdgcn_raw_buffer_load_b32(rsb, tid < RB ? (uint32_t)(n0 + tid) * 4 : kOOB, 0, 0);
    }
  }

  // per-lane parts of the load offsets (row, token, lane group; kOOB for
  // rows >= N); the iteration enters as a wave-uniform soffset. Token rows
  // past M read row M-1: their MFMA rows only feed outputs that are never
  // stored, and in-bounds duplicates cost the address unit far less than
  // masked lanes.
  uint32_t vw[RT], vx[MT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int n = n0 + 16 * t + lr;
    // lane group lg: the codes of K [32 lg, 32 lg + 32) of each iteration
    // (4-bit: 16 bytes, 3-bit: one block of 12)
    vw[t] = n < N ? (uint32_t)n * row_code_bytes<WB>(K) + (WB == 4 ? 16 : 12) * lg : kOOB;
  }
  const bool xl = a.xlds;
  const char* xs = smem;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = min(16 * mt + lr, M - 1);
    vx[mt] = xl ? (uint32_t)m * a.xstride + 64 * lg : ((uint32_t)m * K + 32 * lg) * 2;
  }
  auto load_w = [&](u32x4 (&w)[RT], int it) {
#pragma unroll
    for (int t = 0; t < RT; ++t)
      w[t] = WB == 4 ? bld128s(rq, vw[t], (uint32_t)it * (kIterK / 2))
                     : bld96s(rq, vw[t], (uint32_t)it * (kIterK / 8 * 3));
  };
  // EPI_LOCAL: the block's K-slice of A (16 rows, rows >= r zero) and of
  // w_g (row 16) is staged in LDS with coalesced 16-byte chunks: read in the
  // MFMA lane layout straight from memory, every load would touch 32 cache
  // lines. The MFMAs then take A's rows (lane lr: row lr) and w_g in every
  // column as two further B operands.
  // INT8 A: eight codes (8 bytes) per chunk, staged as exact integers; the
  // rows' scales multiply the fp32 projection sums instead. The thread that
  // reduces column c of the projection tiles always has c = (lane / 4) % 16
  // (the block is a whole number of waves), so it holds that row's scale.
  const rsrc_t ra = kI8 ? make_rsrc(a.ec.A8, (uint32_t)r * K)
                        : make_rsrc(kLoc ? a.ec.A : nullptr, kLoc ? (uint32_t)r * K * 2 : 0u);
  const rsrc_t rgw = make_rsrc(kLoc ? a.ec.wg : nullptr,
                               kLoc && a.ec.gate == GATE_SIGMOID ? (uint32_t)K * 2 : 0u);
  // (a buffer load: a flat load would also hold the LDS counter the
  // prologue's barriers wait on)
  float sa_c = 1.f;
  if constexpr (kI8) {
    const rsrc_t rsa = make_rsrc(a.ec.sa, (uint32_t)r * 4);
    sa_c = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
        rsa, ((lane >> 2) & 15) < r ? (uint32_t)((lane >> 2) & 15) * 4 : kOOB, 0, 0));
  }
  const int acpr = (it_end - it_blk) * (kIterK / 8);  // 16-byte chunks per row
  const int astride = acpr * 8 + 8;                   // LDS row stride (halves)
  uint16_t* als = (uint16_t*)(smem + a.lds_a);        // [17][astride]
  auto a_issue = [&](int base, u32x4 (&c4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ci = base + u * (int)blockDim.x;
      const int row = ci / acpr, kc = ci - row * acpr;
      const bool ok = ci < 16 * acpr && row < r;
      if constexpr (kI8) {
        const u32x2 q = bld64(ra, ok ? (uint32_t)row * K + it_blk * kIterK + 8 * kc : kOOB);
        c4[u] = u32x4{q[0], q[1], 0u, 0u};
      } else {
        c4[u] = bld128(ra, ok ? ((uint32_t)row * K + it_blk * kIterK + 8 * kc) * 2 : kOOB);
      }
    }
  };
  auto a_store = [&](int base, const u32x4 (&c4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ci = base + u * (int)blockDim.x;
      const int row = ci / acpr, kc = ci - row * acpr;
      u32x4 v = c4[u];
      if constexpr (kI8) v = i8x8_exact<DT>(v[0], v[1]);
      if (ci < 16 * acpr) *(u32x4*)(als + row * astride + 8 * kc) = v;
    }
  };
  auto load_x = [&](u32x4 (&xv)[MT][4], int it) {
    if (xl) {
      const uint32_t kb = (uint32_t)(it - it_blk) * (kIterK * 2);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) xv[mt][jj] = *(const u32x4*)(xs + vx[mt] + kb + 16 * jj);
    } else {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          xv[mt][jj] = bld128s(rx, vx[mt] + 16 * jj, (uint32_t)it * (kIterK * 2));
    }
  };

  // Every global load of the prologue is issued before the first wait: the
  // rows of B, the block's slice of x, the scales and zero points, then the
  // first two pipeline stages of codes. Small layers give a wave one or two
  // iterations, so the prologue's round trips are most of the kernel.
  // NST stages of codes in flight per wave: two alternating register sets,
  // or (NST > 2, for long K-slices on wide layers) a ring of NST sets with
  // the activations read right before each iteration (from LDS when staged)
  u32x4 wA[RT], wB[RT];
  u32x4 xA[MT][4], xB[MT][4];
  u32x4 wR[NST > 2 ? NST : 1][RT];
  const int last = iw_end - 1;
  // the block's slice of x into LDS ([M][slice] with a padded row stride),
  // four 16-byte chunks per thread per round
  const int cpr = (it_end - it_blk) * (kIterK / 8);  // 16-byte chunks per row
  const int nch = xl ? M * cpr : 0;
  auto x_issue = [&](int base, u32x4 (&c4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ci = base + u * (int)blockDim.x;
      const int m = ci / cpr, kc = ci - m * cpr;
      c4[u] = bld128(rx, ci < nch ? ((uint32_t)m * K + it_blk * kIterK + 8 * kc) * 2 : kOOB);
    }
  };
  auto x_store = [&](int base, const u32x4 (&c4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int ci = base + u * (int)blockDim.x;
      const int m = ci / cpr, kc = ci - m * cpr;
      if (ci < nch) *(u32x4*)(smem + (size_t)m * a.xstride + 16 * kc) = c4[u];
    }
  };
  // scales and zero points of the block's rows and groups, staged once in
  // LDS with coalesced loads ([row][group] as s | z << 16): per-iteration
  // scattered 2- and 1-byte loads would cost a cache-line request per row
  const int ipg = G / kIterK;  // iterations per quantisation group
  const int g_lo = it_blk / ipg;
  const int ngb = (it_end - 1) / ipg + 1 - g_lo;
  const int ngs = ngb | 1;  // odd LDS row stride: rows fall on distinct banks
  uint32_t* szs = (uint32_t*)(smem + a.lds_sz);
  const int nsz = RB * ngb;
  auto sz_issue = [&](int i0, uint32_t (&sv)[4], uint32_t (&zv)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = i0 + u * (int)blockDim.x;
      const int row = idx / ngb, gg = idx - row * ngb;
      const uint32_t eo = (uint32_t)(n0 + row) * a.ngroups + g_lo + gg;
      const bool ok = idx < nsz && n0 + row < N;
      sv[u] = bld16(rsc, ok ? eo * 2 : kOOB);
      zv[u] = bld8(rz, ok ? eo : kOOB);
    }
  };
  auto sz_store = [&](int i0, const uint32_t (&sv)[4], const uint32_t (&zv)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = i0 + u * (int)blockDim.x;
      if (idx < nsz) {
        const int row = idx / ngb, gg = idx - row * ngb;
        szs[row * ngs + gg] = sv[u] | (zv[u] << 16);
      }
    }
  };
  // eight groups per 16-byte scale load and 8-byte zero load when the
  // block's group range is 8-aligned (2- and 1-byte loads per entry would be
  // a third of the block's load instructions for a few percent of its bytes)
  const bool sz8 = (a.ngroups & 7) == 0 && (g_lo & 7) == 0 && (ngb & 7) == 0;
  const int c8 = ngb >> 3, nsz8 = RB * c8;
  auto sz8_issue = [&](int i, u32x4& s8, u32x2& z8) {
    const int row = i / c8, q = i - row * c8;
    const bool ok = i < nsz8 && n0 + row < N;
    const uint32_t eo = (uint32_t)(n0 + row) * a.ngroups + g_lo + 8 * q;
    s8 = bld128(rsc, ok ? eo * 2 : kOOB);
    z8 = bld64(rz, ok ? eo : kOOB);
  };
  auto sz8_store = [&](int i, const u32x4& s8, const u32x2& z8) {
    if (i < nsz8) {
      const int row = i / c8, q = i - row * c8;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t sv = (s8[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
        const uint32_t zv = (z8[e >> 2] >> (8 * (e & 3))) & 0xFFu;
        szs[row * ngs + 8 * q + e] = sv | (zv << 16);
      }
    }
  };
  {
    const int step = 4 * (int)blockDim.x;
    u32x4 c4[4];
    uint32_t sv[4], zv[4];
    u32x4 s8;
    u32x2 z8;
    // EPI_LOCAL: the first round of A and w_g goes out with the first round
    // of x, scales and zero points, so that the staging costs one round
    // trip. The second round of x and of the 8-group scales goes out with
    // the first too (a deep slice, 28672 wide, needs two), except in the
    // producer-fused variant, whose 22 more VGPRs there would cost it the
    // second workgroup per CU.
    constexpr bool kTwo = EPI != EPI_FUSED;
    u32x4 a0[4], a1[4], gv0;
    u32x4 c4b[4], s8b;
    u32x2 z8b;
    x_issue(tid, c4);
    if constexpr (kTwo) x_issue(tid + step, c4b);
    if (sz8) {
      sz8_issue(tid, s8, z8);
      if constexpr (kTwo) sz8_issue(tid + (int)blockDim.x, s8b, z8b);
    } else {
      sz_issue(tid, sv, zv);
    }
    if constexpr (kLoc) {
      a_issue(tid, a0);
      a_issue(tid + step, a1);
      gv0 = bld128(rgw, tid < acpr ? ((uint32_t)it_blk * kIterK + 8 * tid) * 2 : kOOB);
    }
    // the first code stages go out after the staging loads: the counter
    // retires in order, so the LDS stores below wait only for x, the scales
    // and A (L2-resident after the first workgroups), not for the codes
    // coming from HBM (70B q, k, v as one launch: 17.7 -> 16.9 us)
    if (iw_beg < iw_end) {
      if constexpr (NST > 2) {
#pragma unroll
        for (int q = 0; q < NST; ++q) load_w(wR[q], min(iw_beg + q, last));
      } else {
        load_w(wA, iw_beg);
        if (!xl) load_x(xA, iw_beg);
        load_w(wB, min(iw_beg + 1, last));
        if (!xl) load_x(xB, min(iw_beg + 1, last));
      }
    }
    x_store(tid, c4);
    if constexpr (kTwo) x_store(tid + step, c4b);
    if (sz8) {
      sz8_store(tid, s8, z8);
      if constexpr (kTwo) sz8_store(tid + (int)blockDim.x, s8b, z8b);
    } else {
      sz_store(tid, sv, zv);
    }
    if constexpr (kLoc) {
      a_store(tid, a0);
      a_store(tid + step, a1);
      if (tid < acpr) *(u32x4*)(als + 16 * astride + 8 * tid) = gv0;
    }
    for (int base = tid + (kTwo ? 2 : 1) * step; base < nch; base += step) {
      x_issue(base, c4);
      x_store(base, c4);
    }
    if (sz8) {
      for (int i = tid + (kTwo ? 2 : 1) * (int)blockDim.x; i < nsz8; i += blockDim.x) {
        sz8_issue(i, s8, z8);
        sz8_store(i, s8, z8);
      }
    } else {
      for (int i0 = tid + step; i0 < nsz; i0 += step) {
        sz_issue(i0, sv, zv);
        sz_store(i0, sv, zv);
      }
    }
    if constexpr (kLoc) {
      // the rest of A: two rounds of four chunks per thread in flight; of
      // w_g: one chunk
      for (int base = tid + 2 * step; base < 16 * acpr; base += 2 * step) {
        a_issue(base, a0);
        a_issue(base + step, a1);
        a_store(base, a0);
        a_store(base + step, a1);
      }
      for (int kc = tid + (int)blockDim.x; kc < acpr; kc += blockDim.x) {
        const u32x4 gv = bld128(rgw, ((uint32_t)it_blk * kIterK + 8 * kc) * 2);
        *(u32x4*)(als + 16 * astride + 8 * kc) = gv;
      }
    }
  }
  uint16_t* bs = (uint16_t*)(smem + a.lds_b);
  if (bpre) {
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int ci = tid + c * (int)blockDim.x;
      if (ci < bchunks) *(u32x4*)(bs + 8 * ci) = bst[c];
    }
    if constexpr (kI8) {
      if (tid < RB) ((uint32_t*)((char*)bs + RB * r))[tid] = sbst;
    }
  }
  __syncthreads();
  if (NST == 2 && xl && iw_beg < iw_end) {
    load_x(xA, iw_beg);
    load_x(xB, min(iw_beg + 1, last));
  }

  constexpr float kBias = code_bias<DT>();
  f32x4 acc[RT][MT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint32_t km = opaque_v(0x000F000Fu);
  const uint32_t kg = opaque_v(DT == DT_F16 ? 0x64006400u : 0x43004300u);
  f32x4 eacc[kLocalTiles][MT];
#pragma unroll
  for (int t = 0; t < kLocalTiles; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) eacc[t][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const u32x4 (&w)[RT], const u32x4 (&xv)[MT][4], int it) {
    if constexpr (kLoc) {
      // A x and w_g x: activations (A operand, token rows) times the rows of
      // A / copies of w_g (B operand, one per column) from LDS, accumulated
      // over the wave's chunk
      const int kb = (it - it_blk) * kIterK + 32 * lg;
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const u32x4 af = *(const u32x4*)(als + lr * astride + kb + 8 * jj);
        const u32x4 gf = *(const u32x4*)(als + 16 * astride + kb + 8 * jj);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          eacc[0][mt] = mfma16<DT>(xv[mt][jj], af, eacc[0][mt]);
          eacc[1][mt] = mfma16<DT>(xv[mt][jj], gf, eacc[1][mt]);
        }
      }
    }
    f32x4 xb[MT];
    u32x4 xp[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      xb[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        xb[mt] = mfma16<DT>(xv[mt][jj], ones8<DT>(), xb[mt]);
        // 4-bit codes pair (q_i, q_{i+4}) within a word: the activations
        // follow; 3-bit pairs are in natural order
        xp[mt][jj] = WB == 4 ? pair_like_codes(xv[mt][jj]) : xv[mt][jj];
      }
    }
    const int gg = it / ipg - g_lo;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      u32x4 wd[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        wd[jj] = WB == 4 ? unpack_biased_r(w[t][jj], km, kg) : unpack3_biased(w[t], jj, kg);
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
  // while batch it is computed (two register sets, alternating, both filled
  // by the prologue). Loads past the wave's last iteration re-read that
  // iteration (never computed), so every load is unconditional.
  if (NST > 2 && iw_beg < iw_end) {
    for (int it = iw_beg; it < iw_end; it += NST) {
#pragma unroll
      for (int q = 0; q < NST; ++q) {
        if (it + q < iw_end) {  // uniform
          u32x4 xv[MT][4];
          load_x(xv, it + q);
          compute(wR[q], xv, it + q);
          load_w(wR[q], min(it + q + NST, last));
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  } else if (iw_beg < iw_end) {
    for (int it = iw_beg; it < iw_end; it += 2) {
      compute(wA, xA, it);
      if (it + 1 >= iw_end) break;
      load_w(wA, min(it + 2, last));
      load_x(xA, min(it + 2, last));
      __builtin_amdgcn_sched_barrier(0);
      compute(wB, xB, it + 1);
      load_w(wB, min(it + 3, last));
      load_x(xB, min(it + 3, last));
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if constexpr (kEC) {
    if (!gw && s == 0) ec_wave<DT, MT, RT, EPI>(a, gen, smem, n0, bpre);
  }
  if (xl) __syncthreads();  // the x region is reused below

  // ---- cross-wave reduction (fixed order) into yacc[token][row]; the EC
  // wave's tiles come last
  float* red = (float*)smem;
  float* ered = red + NW * RT * MT * 256;  // EPI_LOCAL: [NW][kLocalTiles][MT] tiles
  if (gw) {
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        *(f32x4*)(red + (((wave * RT + t) * MT + mt) * 64 + lane) * 4) = acc[t][mt];
    if constexpr (kLoc) {
#pragma unroll
      for (int t = 0; t < kLocalTiles; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          *(f32x4*)(ered + (((wave * kLocalTiles + t) * MT + mt) * 64 + lane) * 4) = eacc[t][mt];
    }
  }
  __syncthreads();
  // EPI_LOCAL: this block's [A; w_g] x (its K-slice), u [token][R1p] in LDS
  float* u_loc = (float*)(smem + a.lds_e);
  const int R1 = a.ec.R1, R1p = a.ec.R1p;
  // Without split-K the sums are complete here: each thread that owns u_j of
  // a token also sums that token's gate logit and writes v_j directly
  // (EPI_LOCAL, below), saving a pass and a barrier.
  float* v_loc = u_loc + 16 * MT * R1p;
  const bool v_direct = a.S == 1 && a.ec.gate != GATE_TANH;
  if constexpr (kLoc) {
    // tile 0: column j < r is u_j; tile 1: column 0 is the gate logit w_g x
    for (int e = tid; e < 256 * kLocalTiles * MT; e += blockDim.x) {
      const int tm = e >> 8, rem = e & 255, ln = rem >> 2, i = rem & 3;
      const int t = tm / MT, mt = tm - t * MT;
      const int tok = 16 * mt + 4 * (ln >> 4) + i, c = ln & 15;
      const int j = t == 0 ? (c < r ? c : -1) : (c == 0 && R1 > r ? r : -1);
      if (j < 0 || (v_direct && t != 0)) continue;
      float v = 0.f;
      for (int w = 0; w < NW; ++w) v += ered[(((w * kLocalTiles + t) * MT + mt) * 64 + ln) * 4 + i];
      if constexpr (kI8) {
        if (t == 0) v *= sa_c;  // c == (lane / 4) % 16 here
      }
      if (v_direct) {
        float g = 1.f;
        if (a.ec.gate == GATE_SIGMOID) {
          float zl = 0.f;  // the logit: tile 1, column 0, same token
          for (int w = 0; w < NW; ++w)
            zl += ered[(((w * kLocalTiles + 1) * MT + mt) * 64 + (ln & 48)) * 4 + i];
          const float z = zl + a.ec.b_g;
          g = z >= 0.f ? 1.f / (1.f + __expf(-z)) : __expf(z) / (1.f + __expf(z));
        }
        v_loc[tok * r + j] = a.ec.alpha * g * v;
      } else {
        u_loc[tok * R1p + j] = v;
      }
    }
  }
  float* yacc = (float*)(smem + a.lds_y);
  const float* evs = (const float*)(smem + a.lds_ev);
  const bool add_ev = kEC && s == 0;
  constexpr int YS = RB;  // yacc row stride: [token][RB rows]
  for (int e = tid; e < 256 * RT * MT; e += blockDim.x) {
    const int tm = e >> 8, rem = e & 255, ln = rem >> 2, i = rem & 3;
    const int t = tm / MT, mt = tm - t * MT;
    float v = 0.f;
    for (int w = 0; w < NW; ++w) v += red[(((w * RT + t) * MT + mt) * 64 + ln) * 4 + i];
    if (add_ev) v += evs[((t * MT + mt) * 64 + ln) * 4 + i];
    const int tok = 16 * mt + 4 * (ln >> 4) + i, row = 16 * t + (ln & 15);
    yacc[tok * YS + row] = v;
  }
  __syncthreads();

  // ---- cross-block split-K reduction: the last arriver sums the slices in order
  if (a.S > 1) {
    for (int e = tid; e < RB * M; e += blockDim.x) {
      const int m = e / RB, row = e - m * RB;
      if (n0 + row < N) st_agent(a.ypart + ((size_t)s * M + m) * N + n0 + row, yacc[m * YS + row]);
    }
    if constexpr (kLoc) {
      // the slice's partial [A; w_g] x, for the last arriver of this row
      // group (which waits for this row group's slices only)
      for (int e = tid; e < M * R1; e += blockDim.x) {
        const int m = e / R1, j = e - m * R1;
        st_agent(a.eupart + ((size_t)(rg * a.S + s) * M + m) * R1 + j, u_loc[m * R1p + j]);
      }
    }
    complete_and_sync();
    if (tid == 0) s_flag = arrive_last(a.rb_ctr + rg, (uint32_t)a.S) ? 1 : 0;
    __syncthreads();
    if (!s_flag) {
      if constexpr (EPI == EPI_FUSED) fused_exit(a);
      return;
    }
    // every slice's [M][RB] partial, summed in slice order through the
    // wave-partials region (free now)
    const rsrc_t rp = make_rsrc(a.ypart, (uint32_t)a.S * M * N * 4);
    sum_slices(rp, a.S, M * RB, [&](int q, int i) {
      const int m = i / RB, row = i - m * RB;
      return n0 + row < N ? (uint32_t)(((size_t)q * M + m) * N + n0 + row) * 4u : kOOB;
    }, red, a.lds_y / 4, [&](int i, float v) {
      const int m = i / RB, row = i - m * RB;
      yacc[m * YS + row] = v;
    });
    if constexpr (kLoc) {
      // this row group's slices' [A; w_g] x, summed in slice order
      const rsrc_t re = make_rsrc(a.eupart, (uint32_t)((size_t)a.N / RB + 1) * a.S * M * R1 * 4);
      sum_slices(re, a.S, M * R1, [&](int q, int i) {
        return (uint32_t)(((size_t)(rg * a.S + q) * M) * R1 + i) * 4u;
      }, red, a.lds_y / 4, [&](int i, float v) {
        const int m = i / R1, j = i - m * R1;
        u_loc[m * R1p + j] = v;
      });
    }
  }

  // EPI_LOCAL: v = alpha g(x) (.) A x for every token (g the sigmoid of the
  // gate row's sum plus b_g, or one; or the tanh-MLP gate of u, whose hidden
  // layer takes the LDS after v), then y += v B^T in fp32 below
  if (kLoc && !v_direct && a.ec.gate == GATE_TANH) {
    // LDS after v: the hidden layer (cap x h floats), then the staged
    // parameters when they fit
    float* hid = v_loc + 16 * MT * r;
    const int cap = local_tanh_cap(M, a.ec.h);
    uint16_t* wst = tanh_stage_halves(a.ec.h, r) > 0 ? (uint16_t*)(hid + cap * a.ec.h) : nullptr;
    tanh_gate_tokens<DT>(M, r, a.ec.h, u_loc, R1p, a.ec.W1, a.ec.b1, a.ec.W2, a.ec.b2, a.ec.alpha,
                         hid, cap, v_loc, r, wst);
  } else if (kLoc && !v_direct) {
    for (int idx = tid; idx < M * r; idx += blockDim.x) {
      const int m = idx / r, j = idx - m * r;
      float g = 1.f;
      if (a.ec.gate == GATE_SIGMOID) {
        const float z = u_loc[m * R1p + r] + a.ec.b_g;
        g = z >= 0.f ? 1.f / (1.f + __expf(-z)) : __expf(z) / (1.f + __expf(z));
      }
      v_loc[idx] = a.ec.alpha * g * u_loc[m * R1p + j];
    }
    __syncthreads();
  }
  const uint16_t* bsl = (const uint16_t*)(smem + a.lds_b);

  for (int e = tid; e < RB * M; e += blockDim.x) {
    const int m = e / RB, row = e - m * RB;
    if (n0 + row < N) {
      float v = yacc[m * YS + row];
      if constexpr (kLoc) {
        // v B^T for this row: eight ranks per 16-byte chunk of the staged row
        // of B (r is a multiple of 8 when B is staged), independent loads
        const float* vm = v_loc + m * r;
        float ev = 0.f;
        if (bpre && kI8) {
          // INT8 B staged: the codes and the row's scale exactly, in fp32
          const int8_t* b8row = (const int8_t*)bsl + row * r;
          for (int j0 = 0; j0 < r; j0 += 8) {
            const u32x2 q = *(const u32x2*)(b8row + j0);
            const f32x4 v0 = *(const f32x4*)(vm + j0), v1 = *(const f32x4*)(vm + j0 + 4);
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
              ev += v0[e2] * (float)((int)(q[0] << (24 - 8 * e2)) >> 24);
              ev += v1[e2] * (float)((int)(q[1] << (24 - 8 * e2)) >> 24);
            }
          }
          ev *= ((const float*)((const char*)bsl + RB * r))[row];
        } else if (bpre) {
          for (int j0 = 0; j0 < r; j0 += 8) {
            const u32x4 b8 = *(const u32x4*)(bsl + row * r + j0);
            const f32x4 v0 = *(const f32x4*)(vm + j0), v1 = *(const f32x4*)(vm + j0 + 4);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const float vlo = q < 2 ? v0[2 * q] : v1[2 * q - 4];
              const float vhi = q < 2 ? v0[2 * q + 1] : v1[2 * q - 3];
              ev += vlo * act2f<DT>((uint16_t)(b8[q] & 0xFFFFu)) + vhi * act2f<DT>((uint16_t)(b8[q] >> 16));
            }
          }
        } else if constexpr (kI8) {
          // INT8 B: the codes and the row's scale exactly, in fp32
          const int8_t* br = a.B8 + (size_t)(n0 + row) * r;
          for (int j = 0; j < r; ++j) ev += vm[j] * (float)br[j];
          ev *= a.sb[n0 + row];
        } else {
          const uint16_t* br = a.B + (size_t)(n0 + row) * r;
          for (int j = 0; j < r; ++j) ev += vm[j] * act2f<DT>(br[j]);
        }
        v += ev;
      }
      if (a.res) v += act2f<DT>(res_pre ? resv : a.res[(size_t)m * N + n0 + row]);
      a.y[(size_t)m * N + n0 + row] = f2act<DT>(v);
    }
  }
  if constexpr (EPI == EPI_FUSED) fused_exit(a);
}

// Minimum waves per SIMD the compiler must leave room for (the second
// launch bound). One token tile on up to 32 rows without the local EC asks
// for 4, two workgroups of eight waves per CU (at most 128 VGPRs): wide
// layers run several rounds of blocks, and one block per CU leaves half the
// latency hiding unused (70B gate, fused: 60.8 us at 156 VGPRs, 42.6 us at
// 125).
constexpr int gemv_min_waves(int MT, int RT, int EPI) {
  return MT == 1 && RT <= 2 && EPI <= EPI_FUSED ? 4 : 1;
}

template <int DT, int MT, int RT, int EPI, int WB, int NST>
__global__ __launch_bounds__(kGemvMaxThreads, gemv_min_waves(MT, RT, EPI)) void k_gemv(GemvParams a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  int bid = blockIdx.x;
  uint32_t gen = 0;
  if constexpr (EPI == EPI_FUSED) {
    // the first n_prod workgroups are the EC producers
    gen = (uint32_t)(__hip_atomic_load(gen_counter(a, bid), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >> 32);
    if (bid < a.n_prod) {
      ec_producer<DT, 1>(a.ec, bid, gen, smem);
      fused_exit(a);
      return;
    }
    bid -= a.n_prod;
  }
  gemv_body<DT, MT, RT, EPI, WB, NST>(a, bid, gen, smem);
}

// Several independent layer calls of one GEMV variant in one launch: member i
// owns the workgroups [start[i], start[i+1]) and runs exactly the blocks its
// own launch would run, so each member's output is the one its single call
// writes. The member index is uniform over the workgroup.
template <int DT, int MT, int RT, int EPI, int WB>
__global__ __launch_bounds__(kGemvMaxThreads, gemv_min_waves(MT, RT, EPI)) void k_gemv_group(GemvGroup g) {
  static_assert(EPI == EPI_NONE || EPI == EPI_LOCAL || EPI == EPI_LOCAL_I8,
                "grouped launches take the variants without cross-launch state");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int b = blockIdx.x;
  int i = 0;
#pragma unroll
  for (int j = 1; j < kGroupMax; ++j)
    if (j < g.n && b >= g.start[j]) i = j;
  gemv_body<DT, MT, RT, EPI, WB>(g.p[i], b - g.start[i], 0u, smem);
}

// ---------------------------------------------------------------------------
// Prefill GEMM: 128x128 output tile per block (tokens x rows), K staged 64 at
// a time through double-buffered LDS; the packed codes are dequantised once
// per block into the LDS tile, (q - z) exact then times s with one rounding
// (fp16) or via fp32 (bf16). Four waves, 2x2, each 64x64 = 4x4 MFMA tiles.
// ---------------------------------------------------------------------------
// NP pairs of raw codes (natural K order, one code per 16-bit lane) to
// dequantised act-dtype pairs: (q - z) exact, then one rounding of its
// product with s (fp16: the biased code minus 1024 + z, an exact integer, in
// packed half math; bf16: in fp32, then rounded).
template <int DT, int NP>
__device__ __forceinline__ void dequant_pairs(const uint32_t (&p)[NP], float s, int z,
                                              uint32_t (&out)[NP]) {
  if constexpr (DT == DT_F16) {
    const _Float16 zb = (_Float16)(1024 + z);
    const f16x2 nz = f16x2{-zb, -zb};
    const f16x2 s2 = f16x2{(_Float16)s, (_Float16)s};
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const f16x2 q = __builtin_bit_cast(f16x2, p[i] | 0x64006400u);
      out[i] = __builtin_bit_cast(uint32_t, (q + nz) * s2);
    }
  } else {
    const float zf = (float)z;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const float a0 = ((float)(p[i] & 0xFFFF) - zf) * s;
      const float a1 = ((float)(p[i] >> 16) - zf) * s;
      out[i] = (uint32_t)f2act<DT>(a0) | ((uint32_t)f2act<DT>(a1) << 16);
    }
  }
}

// One packed word of 4-bit codes, dequantised in natural order: pairs
// (q0,q1), (q2,q3), (q4,q5), (q6,q7).
template <int DT>
__device__ __forceinline__ void dequant_word_pairs(uint32_t w, float s, int z, uint32_t (&out)[4]) {
  const uint32_t lo = w & 0x0F0F0F0Fu;         // q0 q2 q4 q6
  const uint32_t hi = (w >> 4) & 0x0F0F0F0Fu;  // q1 q3 q5 q7
  uint32_t p[4];
  p[0] = __builtin_amdgcn_perm(hi, lo, 0x0C040C00u);
  p[1] = __builtin_amdgcn_perm(hi, lo, 0x0C050C01u);
  p[2] = __builtin_amdgcn_perm(hi, lo, 0x0C060C02u);
  p[3] = __builtin_amdgcn_perm(hi, lo, 0x0C070C03u);
  dequant_pairs<DT, 4>(p, s, z, out);
}

// Pairs P0 .. P0 + NP - 1 of a block of 3-bit codes (three words in w),
// dequantised in natural order.
template <int DT, int P0, int NP>
__device__ __forceinline__ void dequant_block3_pairs(const u32x4& w, float s, int z,
                                                     uint32_t (&out)[NP]) {
  uint32_t p[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) p[i] = w3_pair(w, P0 + i, 0u);
  dequant_pairs<DT, NP>(p, s, z, out);
}

// ---------------------------------------------------------------------------
// Dequantisation diagnostic, by the code the prefill GEMM dequantises its
// weight tiles with ((q - z) exact, then one rounding of its product with s):
// one thread per packed word of 4-bit codes (eight outputs), or per block of
// 3-bit codes (three words, 32 outputs).
// ---------------------------------------------------------------------------
template <int DT, int WB>
__global__ __launch_bounds__(256) void k_dequant(const uint32_t* __restrict__ qw,
                                                 const uint16_t* __restrict__ sc,
                                                 const uint8_t* __restrict__ zr,
                                                 uint16_t* __restrict__ out, int N, int K, int G) {
  constexpr int CPU = WB == 4 ? 8 : 32;  // codes per unit (word or block)
  const int kw = K / CPU;
  const long long nunits = (long long)N * kw;
  const long long wi = (long long)blockIdx.x * 256 + threadIdx.x;
  if (wi >= nunits) return;
  const int n = (int)(wi / kw);
  const int k = (int)(wi % kw) * CPU;
  const int ng = K / G;
  const int g = k / G;
  const float s = h2f(sc[(long long)n * ng + g]);
  const int z = zr[(long long)n * ng + g];
  if constexpr (WB == 4) {
    uint32_t o[4];
    dequant_word_pairs<DT>(qw[wi], s, z, o);
    *(u32x4*)(out + (long long)n * K + k) = u32x4{o[0], o[1], o[2], o[3]};
  } else {
    const uint32_t* b = qw + 3 * wi;
    const u32x4 w = u32x4{b[0], b[1], b[2], 0u};
    uint32_t o[16];
    dequant_block3_pairs<DT, 0, 16>(w, s, z, o);
#pragma unroll
    for (int c = 0; c < 4; ++c)
      *(u32x4*)(out + (long long)n * K + k + 8 * c) = u32x4{o[4 * c], o[4 * c + 1], o[4 * c + 2], o[4 * c + 3]};
  }
}

// Split-K tile reduction of the GEMM: a thread's 16 f32x4 of the tile from
// each of the S slices, summed in slice order (slice 0 first, so the result
// does not depend on which slice arrives last). The slices' loads are issued
// in rounds of 32 (S/2 rounds), each round's loads all in flight together:
// the partials sit at the device coherence point, a memory round trip away,
// and one round per slice would pay that latency S times.
// base: byte offset of the thread's first f32x4 in slice 0; slice: bytes
// between slices; entry (i, j) is 1024 * (4i + j) bytes further.
template <int S>
__device__ __forceinline__ void gemm_sum_slices(rsrc_t rp, uint32_t base, uint32_t slice,
                                                f32x4 (&acc)[4][4]) {
  constexpr int E = 32 / S;  // entries per round
#pragma unroll
  for (int rd = 0; rd < S / 2; ++rd) {
    f32x4 pv[S][E];
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int e = 0; e < E; ++e) pv[q][e] = bld128cf(rp, base + q * slice + (rd * E + e) * 1024);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      f32x4 t = pv[0][e];
#pragma unroll
      for (int q = 1; q < S; ++q) t += pv[q][e];
      acc[(rd * E + e) >> 2][(rd * E + e) & 3] = t;
    }
  }
}

// The same for the fully fused variant's EC accumulators: 4 f32x4 per
// thread per slice, all slices' loads in one round (S <= 8: 32 loads).
template <int S>
__device__ __forceinline__ void gemm_sum_ec_slices(rsrc_t rp, uint32_t base, uint32_t slice,
                                                   f32x4 (&eacc)[4]) {
  f32x4 pv[S][4];
#pragma unroll
  for (int q = 0; q < S; ++q)
#pragma unroll
    for (int i = 0; i < 4; ++i) pv[q][i] = bld128cf(rp, base + q * slice + i * 1024);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f32x4 t = pv[0][i];
#pragma unroll
    for (int q = 1; q < S; ++q) t += pv[q][i];
    eacc[i] = t;
  }
}

// TMW: waves along the tokens. TMW = 2: 128-token tiles, 4 waves, two
// workgroups per CU; TMW = 4: 256-token tiles, 8 waves, one workgroup per
// CU. Both keep 64 x 64 per wave and two waves per SIMD; the 256-token tile
// reuses each dequantised weight tile for twice the MFMAs, halving the
// dequantisation's VALU work per MFMA.
template <int DT, int EPI, int TMW, int WB>
__global__ __launch_bounds__(128 * TMW, TMW == 2 ? 2 : 1) void k_gemm(GemmParams a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr bool kLoc = EPI == EPI_LOCAL || EPI == EPI_LOCAL_I8;
  constexpr bool kI8 = EPI == EPI_LOCAL_I8;  // INT8 A and B
  constexpr int TM = 64 * TMW;         // tokens per tile
  constexpr int NT = 128 * TMW;        // threads
  constexpr int WPT = TMW == 2 ? 4 : 2;  // packed words of codes per thread and step
  constexpr int WPR = 8 / WPT;         // threads per row of codes
  constexpr int LR = kGemmLdsRow;
  constexpr int TILEX = TM * LR;       // halves per LDS activation tile
  constexpr int TILEW = kGemmTN * LR;  // halves per LDS weight tile
  constexpr int ETILE = kGemmEcRows * LR;
  uint16_t* Xs = (uint16_t*)smem;             // [2][TM][LR]
  uint16_t* Ws = Xs + 2 * TILEX;              // [2][128][LR]
  uint16_t* Es = Ws + 2 * TILEW;              // EPI_LOCAL: [2][17][LR] A rows, w_g
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int M = a.M, N = a.N, K = a.K;
  const int tiles_m = (M + TM - 1) / TM, tiles_n = (N + kGemmTN - 1) / kGemmTN;
  // Workgroups are dealt to the eight XCDs in turn (b % 8), and each XCD has
  // its own L2: give XCD x a contiguous band of token tiles (or, failing
  // that, of row tiles) so that the tiles its workgroups share are fetched
  // into its L2 once, instead of every activation tile once per XCD.
  // split-K: workgroup b of slice s is blockIdx.x = s * tiles + b
  const int T = tiles_m * tiles_n;
  const int ks = (int)blockIdx.x / T, tb = (int)blockIdx.x - ks * T;
  int mt_i, nt_i;
  {
    const int b = tb, x = b & 7, j = b >> 3;
    if ((tiles_m & 7) == 0) {
      const int pm = tiles_m >> 3;
      mt_i = x * pm + j % pm;
      nt_i = j / pm;
    } else if ((tiles_n & 7) == 0) {
      const int pn = tiles_n >> 3;
      nt_i = x * pn + j % pn;
      mt_i = j / pn;
    } else {
      mt_i = b / tiles_n;
      nt_i = b - mt_i * tiles_n;
    }
  }
  const int m0 = mt_i * TM;
  const int n0 = nt_i * kGemmTN;
  const int KT = K / kGemmTK / a.S;  // steps of this slice (an even count)
  const int kbase = ks * KT;

  // per-thread global load assignments (bounds-checked buffer loads)
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)M * K * 2);
  const rsrc_t rq = make_rsrc(a.qw, (uint32_t)N * row_code_bytes<WB>(K));
  const rsrc_t rsc = make_rsrc(a.sc, (uint32_t)N * a.ngroups * 2);
  const rsrc_t rz = make_rsrc(a.zr, (uint32_t)N * a.ngroups);
  int xr[4], xc[4];
  uint32_t xoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + NT * i;
    xr[i] = c >> 3;
    xc[i] = (c & 7) * 8;
    xoff[i] = m0 + xr[i] < M ? ((uint32_t)(m0 + xr[i]) * K + xc[i]) * 2 : kOOB;
  }
  // codes: row wr, K [8 WPT wp, +8 WPT) of the row's 64-wide step: 4-bit
  // words [wp WPT, +WPT); 3-bit: block wp (WPT = 4) or half wp % 2 of block
  // wp / 2 (WPT = 2), whose three words are loaded whole
  const int wr = tid / WPR, wp = tid % WPR;
  const int wn_row = n0 + wr;
  const bool wok = wn_row < N;
  const uint32_t woff = !wok      ? kOOB
                        : WB == 4 ? (uint32_t)wn_row * (K / 2) + 4 * WPT * wp
                                  : (uint32_t)wn_row * row_code_bytes<WB>(K) + 12 * (WPT == 4 ? wp : wp >> 1);
  // EPI_LOCAL: thread t < 136 stages 16 bytes of the EC tile per step: row
  // t / 8 (A's row while below r, zero up to 15; w_g as row 16), chunk t % 8
  const int er = tid >> 3, ec8 = tid & 7;
  // INT8 A: the chunk's eight codes (8 bytes), dequantised with row er's
  // scale when stored
  const rsrc_t ra = kI8 ? make_rsrc(a.A8, (uint32_t)a.r * K)
                        : make_rsrc(kLoc ? a.A : nullptr, kLoc ? (uint32_t)a.r * K * 2 : 0u);
  const rsrc_t rgw = make_rsrc(kLoc ? a.wg : nullptr,
                               kLoc && a.gate == GATE_SIGMOID ? (uint32_t)K * 2 : 0u);
  const uint32_t eoff = er < 16 && er < a.r ? ((uint32_t)er * K + 8 * ec8) * 2 : kOOB;
  float sa_er = 0.f;
  if constexpr (kI8) {
    const rsrc_t rsa = make_rsrc(a.sa, (uint32_t)a.r * 4);
    sa_er = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
        rsa, er < 16 && er < a.r ? (uint32_t)er * 4 : kOOB, 0, 0));
  }
  const uint32_t goff = er == 16 ? 16u * ec8 : kOOB;

  // two register sets of global loads, so that the loads of step kt+2 are
  // in flight while step kt is computed. The scale and zero point stay raw
  // until the stage is stored: converting them at load time would make the
  // wave wait for every load issued before them (the vector-memory counter
  // retires in order).
  struct Stage {
    u32x4 x[4];
    u32x4 w;
    uint32_t s, z;
    u32x4 e, g;  // EPI_LOCAL: A / w_g chunk, combined when stored
  };
  Stage g0, g1;
  auto gload = [&](Stage& st, int kt) {
    const uint32_t k0 = (uint32_t)(kbase + kt) * kGemmTK;
#pragma unroll
    for (int i = 0; i < 4; ++i) st.x[i] = bld128(rx, xoff[i] + k0 * 2);
    if constexpr (WB == 3) {
      st.w = bld96s(rq, woff, k0 / 8 * 3);
    } else if constexpr (WPT == 4) {
      st.w = bld128(rq, woff + k0 / 2);
    } else {
      const u32x2 q = bld64(rq, woff + k0 / 2);
      st.w = u32x4{q[0], q[1], 0u, 0u};
    }
    const uint32_t g = k0 / a.G;
    st.s = bld16(rsc, wok ? ((uint32_t)wn_row * a.ngroups + g) * 2 : kOOB);
    st.z = bld8(rz, wok ? (uint32_t)wn_row * a.ngroups + g : kOOB);
    if constexpr (kI8) {
      const u32x2 q = bld64(ra, eoff == kOOB ? kOOB : eoff / 2 + k0);
      st.e = u32x4{q[0], q[1], 0u, 0u};
      st.g = bld128(rgw, goff == kOOB ? kOOB : goff + k0 * 2);
    } else if constexpr (kLoc) {
      st.e = bld128(ra, eoff == kOOB ? kOOB : eoff + k0 * 2);
      st.g = bld128(rgw, goff == kOOB ? kOOB : goff + k0 * 2);
    }
  };
  auto lstore = [&](const Stage& st, int buf) {
    const u32x4 (&xreg)[4] = st.x;
    const u32x4 wreg = st.w;
    const float sreg = h2f((uint16_t)st.s);
    const int zreg = (int)st.z;
    uint16_t* xs = Xs + buf * TILEX;
    uint16_t* ws = Ws + buf * TILEW;
#pragma unroll
    for (int i = 0; i < 4; ++i) *(u32x4*)(xs + xr[i] * LR + xc[i]) = xreg[i];
    if constexpr (WB == 4) {
#pragma unroll
      for (int c = 0; c < WPT; ++c) {
        uint32_t o[4];
        dequant_word_pairs<DT>(wreg[c], sreg, zreg, o);
        *(u32x4*)(ws + wr * LR + 8 * (WPT * wp + c)) = u32x4{o[0], o[1], o[2], o[3]};
      }
    } else {
      uint32_t o[4 * WPT];
      if constexpr (WPT == 4) {
        dequant_block3_pairs<DT, 0, 16>(wreg, sreg, zreg, o);
      } else {
        // half 1 of the block: its low fields are word 1, its high bits the
        // upper byte of each half of word 2 (moved down: no branch per lane)
        const bool h1 = (wp & 1) != 0;
        const u32x4 wh = u32x4{h1 ? wreg[1] : wreg[0], 0u, h1 ? wreg[2] >> 8 : wreg[2], 0u};
        dequant_block3_pairs<DT, 0, 8>(wh, sreg, zreg, o);
      }
#pragma unroll
      for (int c = 0; c < WPT; ++c)
        *(u32x4*)(ws + wr * LR + 8 * (WPT * wp + c)) = u32x4{o[4 * c], o[4 * c + 1], o[4 * c + 2], o[4 * c + 3]};
    }
    if constexpr (kLoc) {
      u32x4 ev = st.e;
      if constexpr (kI8) ev = i8x8_to_act<DT>(ev[0], ev[1], sa_er);
      if (tid < kGemmEcRows * 8) *(u32x4*)(Es + buf * ETILE + er * LR + 8 * ec8) = ev | st.g;
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // EPI_LOCAL: u = x A^T (waves of row half 0) and the gate logit x w_g
  // (row half 1, w_g in every column) for the wave's 64 tokens
  f32x4 eacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) eacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const uint16_t* xs = Xs + buf * TILEX;
    const uint16_t* ws = Ws + buf * TILEW;
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
      if constexpr (kLoc) {
        const u32x4 ef = *(const u32x4*)(Es + buf * ETILE + (wn == 0 ? lr : 16) * LR + kk + 8 * lg);
#pragma unroll
        for (int i = 0; i < 4; ++i) eacc[i] = mfma16<DT>(af[i], ef, eacc[i]);
      }
    }
  };

  // Step kt computes LDS buffer kt & 1. Its loads were issued two steps
  // earlier into register set kt & 1, and it is stored at the start of its
  // step while the next step's loads are still in flight. K is a multiple of
  // 128, so the steps come in pairs and the loop has a single exit; loads
  // past the last step re-read it (never stored), so that every load is
  // unconditional. Both ways into the loop head thus leave the same loads in
  // flight, and the wait before a store covers only the stage being stored.
  // One barrier per step: a buffer is rewritten only after every wave has
  // passed the barrier that follows its last read.
  const int kl = KT - 1;
  gload(g0, 0);
  __builtin_amdgcn_sched_barrier(0);
  gload(g1, 1);
  __builtin_amdgcn_sched_barrier(0);
  for (int kt = 0; kt < KT; kt += 2) {
    lstore(g0, 0);
    __syncthreads();
    gload(g0, min(kt + 2, kl));
    __builtin_amdgcn_sched_barrier(0);
    compute(0);
    __builtin_amdgcn_sched_barrier(0);
    lstore(g1, 1);
    __syncthreads();
    gload(g1, min(kt + 3, kl));
    __builtin_amdgcn_sched_barrier(0);
    compute(1);
    __builtin_amdgcn_sched_barrier(0);
  }

  // split-K: every slice publishes its tile (lane-major f32x4), and with
  // EPI_LOCAL its EC accumulators; the last to arrive sums the slices in
  // slice order (reading its own back like the others) and runs the epilogue
  if (a.S > 1) {
    __shared__ int s_last;
    const uint32_t tbytes = TM * kGemmTN * 4;
    const rsrc_t rp = make_rsrc(a.ypart, (uint32_t)a.S * T * tbytes);
    const uint32_t ybase = (uint32_t)tb * tbytes + (uint32_t)(wave * 16 * 64 + lane) * 16;
    const uint32_t yslice = (uint32_t)T * tbytes;
    constexpr uint32_t ebytes = 2 * TMW * 4 * 64 * 16;  // EC accumulators of a tile
    const rsrc_t rep = make_rsrc(kLoc ? a.epart : nullptr, kLoc ? (uint32_t)a.S * T * ebytes : 0u);
    const uint32_t ebase = (uint32_t)tb * ebytes + (uint32_t)(wave * 4 * 64 + lane) * 16;
    const uint32_t eslice = (uint32_t)T * ebytes;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) bst128c(rp, ybase + ks * yslice + (i * 4 + j) * 1024, acc[i][j]);
    if constexpr (kLoc) {
#pragma unroll
      for (int i = 0; i < 4; ++i) bst128c(rep, ebase + ks * eslice + i * 1024, eacc[i]);
    }
    complete_and_sync();
    if (tid == 0) s_last = arrive_last(a.ctr + tb, (uint32_t)a.S) ? 1 : 0;
    __syncthreads();
    if (!s_last) return;
    if (a.S == 2) {
      gemm_sum_slices<2>(rp, ybase, yslice, acc);
      if constexpr (kLoc) gemm_sum_ec_slices<2>(rep, ebase, eslice, eacc);
    } else if (a.S == 4) {
      gemm_sum_slices<4>(rp, ybase, yslice, acc);
      if constexpr (kLoc) gemm_sum_ec_slices<4>(rep, ebase, eslice, eacc);
    } else {
      gemm_sum_slices<8>(rp, ybase, yslice, acc);
      if constexpr (kLoc) gemm_sum_ec_slices<8>(rep, ebase, eslice, eacc);
    }
  }

  // EPI_LOCAL: v = alpha g(x) (.) u for the block's TM tokens, as act-dtype
  // high and low parts [TM][32] in LDS (the stage buffers are free once
  // every wave is past its last step)
  constexpr int kVS = 32;
  float* u_sh = (float*)smem;                                  // [TM][17]
  uint16_t* vh_sh = (uint16_t*)(smem + TM * 17 * 4);           // [TM][kVS]
  uint16_t* vl_sh = vh_sh + TM * kVS;
  if constexpr (kLoc) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        const int t = wm * 64 + 16 * i + 4 * lg + e2;
        if (wn == 0 && lr < a.r) u_sh[t * 17 + lr] = eacc[i][e2];
        if (wn == 1 && lr == 0) u_sh[t * 17 + 16] = eacc[i][e2];
      }
    __syncthreads();
    // the tanh-MLP gate: v [TM][16] in fp32 first, its hidden layer in the
    // rest of the (free) stage buffers
    float* v_sh = (float*)(smem + TM * 17 * 4 + 2 * TM * kVS * 2);
    const bool tanh_g = a.gate == GATE_TANH;  // uniform
    if (tanh_g) {
      // after v: the staged parameters (when they fit), then the hidden layer
      constexpr int kLds = 2 * (TM + kGemmTN) * LR * 2 + 2 * kGemmEcRows * LR * 2;
      const int nst = tanh_stage_halves(a.h, a.r);
      uint16_t* wst = nst > 0 ? (uint16_t*)(v_sh + TM * 16) : nullptr;
      float* hid = (float*)((char*)(v_sh + TM * 16) + align_up((size_t)nst * 2, 16));
      const int hid_floats = (kLds - (int)((char*)hid - smem)) / 4;
      const int cap = max(1, min(TM, hid_floats / max(1, a.h)));
      tanh_gate_tokens<DT>(TM, a.r, a.h, u_sh, 17, a.W1, a.b1, a.W2, a.b2, a.alpha, hid, cap,
                           v_sh, 16, wst);
    }
    for (int idx = tid; idx < TM * kVS; idx += NT) {
      const int t = idx / kVS, j = idx - t * kVS;
      float val = 0.f;
      if (j < a.r && tanh_g) {
        val = v_sh[t * 16 + j];
      } else if (j < a.r) {
        float g = 1.f;
        if (a.gate == GATE_SIGMOID) {
          const float z = u_sh[t * 17 + 16] + a.b_g;
          g = z >= 0.f ? 1.f / (1.f + __expf(-z)) : __expf(z) / (1.f + __expf(z));
        }
        val = a.alpha * g * u_sh[t * 17 + j];
      }
      const uint16_t hi = f2act<DT>(val);
      vh_sh[idx] = hi;
      vl_sh[idx] = f2act<DT>(val - act2f<DT>(hi));
    }
    __syncthreads();
  }

  if constexpr (EPI == EPI_READY || kLoc) {
    // y += v_hi B^T + v_lo B^T over the rank (zero-padded to vstride); INT8
    // B rows are dequantised with their scale
    const int r = a.r;
    const bool bvec = (r & 7) == 0;
    const bool b8 = kI8 || (EPI == EPI_READY && a.B8 != nullptr);  // uniform
    const int vstride = kLoc ? kVS : a.vstride;
    for (int kr = 0; kr < vstride; kr += 32) {
      const int kk = kr + 8 * lg;
      u32x4 vhf[4], vlf[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = wm * 64 + 16 * i + lr, m = m0 + t;
        const bool ok = m < M;
        if constexpr (kLoc) {
          vhf[i] = *(const u32x4*)(vh_sh + t * kVS + kk);
          vlf[i] = *(const u32x4*)(vl_sh + t * kVS + kk);
        } else {
          vhf[i] = ok ? ldg16(a.vh + (size_t)m * a.vstride + kk) : u32x4{0, 0, 0, 0};
          vlf[i] = ok ? ldg16(a.vl + (size_t)m * a.vstride + kk) : u32x4{0, 0, 0, 0};
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + 16 * j + lr;
        u32x4 f = u32x4{0, 0, 0, 0};
        if (n < N && b8) {
          const int8_t* br = a.B8 + (size_t)n * r;
          const float sb = a.sb[n];
          if (bvec) {
            if (kk < r) {
              const u32x2 q = *(const u32x2*)(br + kk);
              f = i8x8_to_act<DT>(q[0], q[1], sb);
            }
          } else {
            uint32_t h[8];
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2) h[e2] = (kk + e2 < r) ? i8_to_act<DT>(br[kk + e2], sb) : 0u;
            f = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
          }
        } else if (n < N) {
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
        if (m < M) {
          float v = acc[i][j][e2];
          if (a.res) v += act2f<DT>(a.res[(size_t)m * N + n]);
          a.y[(size_t)m * N + n] = f2act<DT>(v);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Prefill GEMM with loading and multiplying waves (4-bit codes, 256 x 128
// tiles, one K-slice; the plain and the semi-fused epilogue). In k_gemm every
// wave dequantises its share of the next step and then multiplies, and the
// step's barrier lines the waves up, so a SIMD runs the dequantisation's
// VALU work and the MFMAs one after the other. Here waves 0-3 only multiply
// (each owns 128 tokens x 64 rows: 8 x 4 MFMA tiles) and waves 4-7 only load:
// they dequantise and store step kt+1's tiles into the free LDS buffer while
// the multiplying waves read step kt's, and issue the loads of step kt+3.
// Each SIMD holds one loading wave beside its multiplying ones, so the two
// streams overlap; one barrier per step. A wave also reads 12 fragments per
// 32 MFMAs here, not 16.
// TNB = 1: 256 x 128 tiles, four multiplying waves (one per SIMD);
// TNB = 2: 256 x 256 tiles, eight multiplying waves (two per SIMD, 144 KB
// of LDS), twelve waves in all, at most 168 registers each.
// WB: code width (4, or 3: three words per 32 codes).
// ---------------------------------------------------------------------------
template <int DT, int EPI, int TNB, int WB>
__global__ __launch_bounds__(256 * (1 + TNB), 1) void k_gemm_ws(GemmParams a) {
  static_assert(EPI == EPI_NONE || EPI == EPI_READY, "plain and semi-fused epilogues");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int TM = 256, TN = kGemmTN * TNB, LR = kGemmLdsRow;
  constexpr int TILEX = TM * kGemmTK, TILEW = TN * LR;
  constexpr int NCW = 4 * TNB;   // multiplying waves: 2 along the tokens, 2 TNB along the rows
  constexpr int WPT = 4 * TNB;   // code words per loading thread and step
  // activations: [2][TM][64] unpadded, the 16-byte chunk c of row t at
  // chunk c ^ (t % 8) (conflict-free fragment reads without padding, which
  // the 1 KB runs of the direct loads below cannot skip)
  uint16_t* Xs = (uint16_t*)smem;
  uint16_t* Ws = Xs + 2 * TILEX;   // [2][TN][LR]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int M = a.M, N = a.N, K = a.K;
  const int tiles_m = (M + TM - 1) / TM, tiles_n = (N + TN - 1) / TN;
  // XCD banding as in k_gemm
  int mt_i, nt_i;
  {
    const int b = (int)blockIdx.x, x = b & 7, j = b >> 3;
    if ((tiles_m & 7) == 0) {
      const int pm = tiles_m >> 3;
      mt_i = x * pm + j % pm;
      nt_i = j / pm;
    } else if ((tiles_n & 7) == 0) {
      const int pn = tiles_n >> 3;
      nt_i = x * pn + j % pn;
      mt_i = j / pn;
    } else {
      mt_i = b / tiles_n;
      nt_i = b - mt_i * tiles_n;
    }
  }
  const int m0 = mt_i * TM, n0 = nt_i * TN;
  const int KT = K / kGemmTK;  // steps (K is a multiple of 128: an even count)

  // EPI_READY: v_hi, v_lo [TM][64] and B [TN][64] (act dtype, zero past the
  // rank, INT8 rows dequantised with their scale) for rank columns
  // kr0 .. kr0 + 63, staged into LDS (free after the K loop) by all waves
  constexpr int ER = 72;  // padded LDS row (halves)
  uint16_t* vhs = (uint16_t*)smem;  // [TM][ER]
  uint16_t* vls = vhs + TM * ER;    // [TM][ER]
  uint16_t* bss = vls + TM * ER;    // [TN][ER]
  auto ec_stage = [&](int kr0) {
    const int r = a.r;
    for (int c = tid; c < 2 * TM * 8; c += 256 * (1 + TNB)) {
      const int lo = c >= TM * 8, cc = lo ? c - TM * 8 : c;
      const int t = cc >> 3, col = kr0 + (cc & 7) * 8, m = m0 + t;
      u32x4 v = u32x4{0, 0, 0, 0};
      if (m < M && col < a.vstride) v = ldg16((lo ? a.vl : a.vh) + (size_t)m * a.vstride + col);
      *(u32x4*)((lo ? vls : vhs) + t * ER + (cc & 7) * 8) = v;
    }
    for (int c = tid; c < TN * 8; c += 256 * (1 + TNB)) {
      const int row = c >> 3, col = kr0 + (c & 7) * 8, n = n0 + row;
      u32x4 f = u32x4{0, 0, 0, 0};
      if (n < N && col < r) {
        if (a.B8) {
          const int8_t* br = a.B8 + (size_t)n * r;
          const float sb = a.sb[n];
          if ((r & 7) == 0) {
            const u32x2 q = *(const u32x2*)(br + col);
            f = i8x8_to_act<DT>(q[0], q[1], sb);
          } else {
            uint32_t h[8];
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2) h[e2] = col + e2 < r ? i8_to_act<DT>(br[col + e2], sb) : 0u;
            f = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
          }
        } else {
          const uint16_t* br = a.B + (size_t)n * r;
          if ((r & 7) == 0) {
            f = ldg16(br + col);
          } else {
            uint32_t h[8];
#pragma unroll
            for (int e2 = 0; e2 < 8; ++e2) h[e2] = col + e2 < r ? br[col + e2] : 0u;
            f = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
          }
        }
      }
      *(u32x4*)(bss + row * ER + (c & 7) * 8) = f;
    }
  };

  if (wave >= NCW) {
    // ---- loading waves: thread pt stages, of each 64-wide step, the codes
    // of K half pt % 2 of row pt / 2 (TNB = 1) or both halves of row pt
    // (TNB = 2): per half four words, or one 3-bit block of three
    const int pt = tid - 64 * NCW;
    const rsrc_t rq = make_rsrc(a.qw, (uint32_t)N * row_code_bytes<WB>(K));
    const rsrc_t rsc = make_rsrc(a.sc, (uint32_t)N * a.ngroups * 2);
    const rsrc_t rz = make_rsrc(a.zr, (uint32_t)N * a.ngroups);
    const int wr = TNB == 2 ? pt : pt >> 1, wp = TNB == 2 ? 0 : pt & 1;
    const int wn_row = n0 + wr;
    const bool wok = wn_row < N;
    const uint32_t woff = !wok ? kOOB : (uint32_t)wn_row * row_code_bytes<WB>(K) + (WB == 4 ? 16 : 12) * wp;
    struct Stage {
      u32x4 w[TNB];
      uint32_t s, z;
    };
    Stage g0, g1;
    auto gload = [&](Stage& st, int kt) {
      const uint32_t k0 = (uint32_t)kt * kGemmTK;
#pragma unroll
      for (int h = 0; h < TNB; ++h) {
        if constexpr (WB == 4) st.w[h] = bld128(rq, wok ? woff + k0 / 2 + 16 * h : kOOB);
        else st.w[h] = bld96s(rq, woff, k0 / 8 * 3 + 12 * h);
      }
      const uint32_t g = k0 / a.G;
      st.s = bld16(rsc, wok ? ((uint32_t)wn_row * a.ngroups + g) * 2 : kOOB);
      st.z = bld8(rz, wok ? (uint32_t)wn_row * a.ngroups + g : kOOB);
    };
    auto lstore = [&](const Stage& st, int buf) {
      uint16_t* ws = Ws + buf * TILEW;
      const float sreg = h2f((uint16_t)st.s);
      const int zreg = (int)st.z;
      if constexpr (WB == 4) {
#pragma unroll
        for (int c = 0; c < WPT; ++c) {
          uint32_t o[4];
          dequant_word_pairs<DT>(st.w[c >> 2][c & 3], sreg, zreg, o);
          *(u32x4*)(ws + wr * LR + 8 * (4 * wp + c)) = u32x4{o[0], o[1], o[2], o[3]};
        }
      } else {
#pragma unroll
        for (int h = 0; h < TNB; ++h) {
          uint32_t o[16];
          dequant_block3_pairs<DT, 0, 16>(st.w[h], sreg, zreg, o);
#pragma unroll
          for (int c = 0; c < 4; ++c)
            *(u32x4*)(ws + wr * LR + 8 * (4 * (wp + h) + c)) =
                u32x4{o[4 * c], o[4 * c + 1], o[4 * c + 2], o[4 * c + 3]};
        }
      }
    };
    // step kt stores step kt + 1 (loaded two steps earlier) and then loads
    // step kt + 3 into the same registers; loads past the end re-read the
    // last step (never stored), so that every load is unconditional
    const int kl = KT - 1;
    gload(g0, 0);
    __builtin_amdgcn_sched_barrier(0);
    gload(g1, min(1, kl));
    __builtin_amdgcn_sched_barrier(0);
    lstore(g0, 0);
    gload(g0, min(2, kl));
    __syncthreads();
    for (int kt = 0; kt < KT; kt += 2) {
      lstore(g1, 1);
      gload(g1, min(kt + 3, kl));
      __syncthreads();
      if (kt + 2 < KT) {
        lstore(g0, 0);
        gload(g0, min(kt + 4, kl));
      }
      __syncthreads();
    }
    if constexpr (EPI == EPI_READY) {
      for (int kr0 = 0; kr0 < a.vstride; kr0 += 64) {
        ec_stage(kr0);
        __syncthreads();
        __syncthreads();
      }
    }
    return;
  }

  // ---- multiplying waves: wave c owns tokens 128 (c / (2 TNB)) .., rows
  // 64 (c % (2 TNB)) .., as 4 x 2 tiles of the 32 x 32 x 16 MFMA (half the
  // MFMA instructions of 16 x 16 x 32 tiles for the same LDS reads: measured
  // alone with the stage stores, 60% of the peak against 51%). They issue
  // ahead of the loading wave of their SIMD when both are ready: the loading
  // waves have a step of slack, the MFMA pipe none.
  __builtin_amdgcn_s_setprio(1);
  const int l32 = lane & 31, lh = lane >> 5;
  const int wm = wave / (2 * TNB), wn = wave % (2 * TNB);
  constexpr int FM32 = 4, FN32 = 2;
  // The activation tile goes straight from memory into LDS (16-byte buffer
  // loads to LDS): the multiplying waves issue it, one step ahead into the
  // free buffer, and wait for it only at the step's barrier, behind their
  // own MFMAs; they have no other memory loads, so the wait covers nothing
  // else. Wave w writes the 1 KB runs w IPW .. +IPW of the tile (eight rows
  // each); lane l of a run lands at 16 l: row 8 run + l / 8, stored chunk
  // l % 8, which holds the row's chunk (l % 8) ^ (row % 8).
  constexpr int IPW = 32 / NCW;  // 1 KB runs per multiplying wave and step
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)M * K * 2);
  uint32_t xoff[IPW];
#pragma unroll
  for (int u = 0; u < IPW; ++u) {
    const int row = (wave * IPW + u) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ (row & 7);
    xoff[u] = m0 + row < M ? ((uint32_t)(m0 + row) * K + 8 * c) * 2 : kOOB;
  }
  auto xdma = [&](int kt, int buf) {
    const uint32_t kb = (uint32_t)kt * kGemmTK * 2;
#pragma unroll
    for (int u = 0; u < IPW; ++u)
      bld128_lds(rx, Xs + buf * TILEX + (wave * IPW + u) * 512, xoff[u] == kOOB ? kOOB : xoff[u] + kb);
  };
  f32x16 acc[FM32][FN32];
#pragma unroll
  for (int i = 0; i < FM32; ++i)
#pragma unroll
    for (int j = 0; j < FN32; ++j) acc[i][j] = f32x16{};
  // 16-K slices: the slice's six fragments, then its eight MFMAs; SW: the
  // token operand is the swizzled activation tile (rows of 64 halves). The
  // scheduling groups keep the reads ahead: the weight fragments and the
  // first two token fragments go out before the first MFMA, then each pair
  // of MFMAs is followed by the next token fragment's read.
  auto mma = [&](const uint16_t* xs, const uint16_t* ws, int xr0, int wr0, int ld, int kk, bool sw) {
    u32x4 bf[FN32], af[FM32];
#pragma unroll
    for (int j = 0; j < FN32; ++j) bf[j] = *(const u32x4*)(ws + (wr0 + 32 * j + l32) * ld + kk + 8 * lh);
#pragma unroll
    for (int i = 0; i < FM32; ++i) {
      const int t = xr0 + 32 * i + l32;
      af[i] = sw ? *(const u32x4*)(xs + t * kGemmTK + 8 * (((kk >> 3) + lh) ^ (t & 7)))
                 : *(const u32x4*)(xs + t * ld + kk + 8 * lh);
    }
#pragma unroll
    for (int i = 0; i < FM32; ++i)
#pragma unroll
      for (int j = 0; j < FN32; ++j) acc[i][j] = mfma32<DT>(af[i], bf[j], acc[i][j]);
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // 4 LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // 2 MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };
  xdma(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // one copy of the step's MFMAs in the loop (two copies, one per buffer,
  // make the register allocator shuffle accumulators between them)
  for (int kt = 0; kt < KT; ++kt) {
    if (kt + 1 < KT) xdma(kt + 1, (kt + 1) & 1);
    const uint16_t* xs = Xs + (kt & 1) * TILEX;
    const uint16_t* ws = Ws + (kt & 1) * TILEW;
#pragma unroll
    for (int kk = 0; kk < kGemmTK; kk += 16) mma(xs, ws, wm * 128, wn * 64, LR, kk, true);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's share of the next tile is in LDS
    __syncthreads();
  }

  if constexpr (EPI == EPI_READY) {
    // y += v_hi B^T + v_lo B^T over the rank (zero-padded to vstride), 64
    // rank columns at a time from LDS, as 32 x 32 x 16 MFMAs like the K loop
    for (int kr0 = 0; kr0 < a.vstride; kr0 += 64) {
      ec_stage(kr0);
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < 64; kk += 16) {
        if (kr0 + kk < a.vstride) {
          mma(vhs, bss, wm * 128, wn * 64, ER, kk, false);
          mma(vls, bss, wm * 128, wn * 64, ER, kk, false);
        }
      }
      __syncthreads();
    }
  }

#pragma unroll
  for (int i = 0; i < FM32; ++i)
#pragma unroll
    for (int j = 0; j < FN32; ++j) {
      const int n = n0 + wn * 64 + 32 * j + l32;
      if (n >= N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm * 128 + 32 * i + 8 * (e >> 2) + 4 * lh + (e & 3);
        if (m < M) {
          float v = acc[i][j][e];
          if (a.res) v += act2f<DT>(a.res[(size_t)m * N + n]);
          a.y[(size_t)m * N + n] = f2act<DT>(v);
        }
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

hipError_t SPEAR_W(launch_dequant)(int dt, const uint32_t* qw, const uint16_t* sc, const uint8_t* zr,
                                   uint16_t* out, int N, int K, int G, hipStream_t st) {
  const long long nunits = (long long)N * (K / (SPEAR_WB == 4 ? 8 : 32));
  const unsigned grid = (unsigned)((nunits + 255) / 256);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, hipLaunchKernelGGL((k_dequant<DTC, SPEAR_WB>), dim3(grid), dim3(256), 0, st,
                                         qw, sc, zr, out, N, K, G));
  return hipGetLastError();
}

#if SPEAR_WB == 4

hipError_t launch_ec(int dt, const EcParams& e, int grid, int block, int ipp, size_t lds,
                     hipStream_t st) {
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, {
    if (ipp == 1) {
      hipError_t err = allow_lds(k_ec<DTC, 1>, lds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL((k_ec<DTC, 1>), dim3(grid), dim3(block), lds, st, e);
    } else {
      hipError_t err = allow_lds(k_ec<DTC, 2>, lds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL((k_ec<DTC, 2>), dim3(grid), dim3(block), lds, st, e);
    }
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

hipError_t launch_rmsnorm(int dt, const uint16_t* y, const uint16_t* w, float eps, uint16_t* y_norm,
                          int M, int N, hipStream_t st) {
  if (M == 0 || N == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, hipLaunchKernelGGL(k_rmsnorm<DTC>, dim3(M), dim3(256), 0, st, y, w, eps,
                                         y_norm, N));
  return hipGetLastError();
}

hipError_t launch_ec_up_acc(int dt, const float* v, const uint16_t* B, const int8_t* B8,
                            const float* sb, uint16_t* y, int M, int N, int r, hipStream_t st) {
  const long long total = (long long)M * N;
  const unsigned grid = (unsigned)((total + 255) / 256);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, hipLaunchKernelGGL(k_ec_up_acc<DTC>, dim3(grid), dim3(256), 0, st, v, B, B8,
                                         sb, y, M, N, r));
  return hipGetLastError();
}

#endif  // SPEAR_WB == 4

template <int DT, int MT, int RT, int EPI, int NST>
static hipError_t gemv_launch_one(const GemvParams& p, int grid, int block, size_t lds,
                                  hipStream_t st) {
  hipError_t err = allow_lds(k_gemv<DT, MT, RT, EPI, SPEAR_WB, NST>, lds);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI, SPEAR_WB, NST>), dim3(grid), dim3(block), lds, st, p);
  return hipGetLastError();
}

// Pipeline depths compiled in: 2 everywhere; 4 for one token tile on the
// variants wide layers take at decode (4-bit only, fused, semi-fused).
template <int DT, int MT, int RT, int EPI>
static hipError_t gemv_launch_nst(int nst, const GemvParams& p, int grid, int block, size_t lds,
                                  hipStream_t st) {
  if constexpr (MT == 1 && (EPI == EPI_NONE || EPI == EPI_READY || EPI == EPI_FUSED)) {
    if (nst == 4) return gemv_launch_one<DT, MT, RT, EPI, 4>(p, grid, block, lds, st);
  }
  if (nst != 2) return hipErrorInvalidValue;
  return gemv_launch_one<DT, MT, RT, EPI, 2>(p, grid, block, lds, st);
}

template <int DT, int MT, int RT>
static hipError_t gemv_launch(int epi, int nst, const GemvParams& p, int grid, int block,
                              size_t lds, hipStream_t st) {
  switch (epi) {
    case EPI_NONE: return gemv_launch_nst<DT, MT, RT, EPI_NONE>(nst, p, grid, block, lds, st);
    case EPI_READY: return gemv_launch_nst<DT, MT, RT, EPI_READY>(nst, p, grid, block, lds, st);
    case EPI_FUSED: return gemv_launch_nst<DT, MT, RT, EPI_FUSED>(nst, p, grid, block, lds, st);
    case EPI_LOCAL: return gemv_launch_nst<DT, MT, RT, EPI_LOCAL>(nst, p, grid, block, lds, st);
    default: return gemv_launch_nst<DT, MT, RT, EPI_LOCAL_I8>(nst, p, grid, block, lds, st);
  }
}

// The GEMV shapes compiled in: (token tiles MT, row tiles RT).
// gemv_shape_supported() mirrors this list for the planner.
#define SPEAR_GEMV_SHAPES(X) \
  X(1, 1) X(1, 2) X(1, 4) X(2, 1) X(2, 2) X(2, 4) X(3, 1) X(3, 2) X(4, 1)

#if SPEAR_WB == 4
bool gemv_shape_supported(int MT, int RT) {
#define SPEAR_GEMV_MATCH(mt, rt) if (MT == mt && RT == rt) return true;
  SPEAR_GEMV_SHAPES(SPEAR_GEMV_MATCH)
#undef SPEAR_GEMV_MATCH
  return false;
}
#endif

hipError_t SPEAR_W(launch_gemv)(int dt, int MT, int RT, int epi, int nst, const GemvParams& p,
                                int grid, int block, size_t lds, hipStream_t st) {
  // split-K needs its partial sums and row-group counters (workspace)
  const bool loc = epi == EPI_LOCAL || epi == EPI_LOCAL_I8;
  if (p.S < 1 || (p.S > 1 && (!p.ypart || !p.rb_ctr || (loc && !p.eupart))) ||
      (epi == EPI_LOCAL_I8 && (!p.ec.A8 || !p.ec.sa || !p.B8 || !p.sb)))
    return hipErrorInvalidValue;
  if (grid == 0) return hipSuccess;
#define SPEAR_GEMV_CASE(mt, rt)                                                     \
  if (MT == mt && RT == rt)                                                         \
    return dt == DT_F16 ? gemv_launch<DT_F16, mt, rt>(epi, nst, p, grid, block, lds, st) \
                        : gemv_launch<DT_BF16, mt, rt>(epi, nst, p, grid, block, lds, st);
  SPEAR_GEMV_SHAPES(SPEAR_GEMV_CASE)
#undef SPEAR_GEMV_CASE
  return hipErrorInvalidValue;
}

template <int DT, int MT, int RT>
static hipError_t gemv_group_launch(int epi, const GemvGroup& g, int block, size_t lds,
                                    hipStream_t st) {
  constexpr int WB = SPEAR_WB;
  const int grid = g.start[g.n];
  hipError_t err = epi == EPI_NONE    ? allow_lds(k_gemv_group<DT, MT, RT, EPI_NONE, WB>, lds)
                   : epi == EPI_LOCAL ? allow_lds(k_gemv_group<DT, MT, RT, EPI_LOCAL, WB>, lds)
                                      : allow_lds(k_gemv_group<DT, MT, RT, EPI_LOCAL_I8, WB>, lds);
  if (err != hipSuccess) return err;
  if (epi == EPI_NONE)
    hipLaunchKernelGGL((k_gemv_group<DT, MT, RT, EPI_NONE, WB>), dim3(grid), dim3(block), lds, st, g);
  else if (epi == EPI_LOCAL)
    hipLaunchKernelGGL((k_gemv_group<DT, MT, RT, EPI_LOCAL, WB>), dim3(grid), dim3(block), lds, st, g);
  else
    hipLaunchKernelGGL((k_gemv_group<DT, MT, RT, EPI_LOCAL_I8, WB>), dim3(grid), dim3(block), lds, st,
                       g);
  return hipGetLastError();
}

hipError_t SPEAR_W(launch_gemv_group)(int dt, int MT, int RT, int epi, const GemvGroup& g,
                                      int block, size_t lds, hipStream_t st) {
  if (g.n < 1 || g.n > kGroupMax || g.start[0] != 0 ||
      (epi != EPI_NONE && epi != EPI_LOCAL && epi != EPI_LOCAL_I8))
    return hipErrorInvalidValue;
  const bool loc = epi == EPI_LOCAL || epi == EPI_LOCAL_I8;
  for (int i = 0; i < g.n; ++i) {
    const GemvParams& p = g.p[i];
    if (g.start[i + 1] < g.start[i] || p.S < 1 ||
        (p.S > 1 && (!p.ypart || !p.rb_ctr || (loc && !p.eupart))) ||
        (epi == EPI_LOCAL_I8 && (!p.ec.A8 || !p.ec.sa || !p.B8 || !p.sb)))
      return hipErrorInvalidValue;
  }
  if (g.start[g.n] == 0) return hipSuccess;
#define SPEAR_GEMV_GROUP_CASE(mt, rt)                                                  \
  if (MT == mt && RT == rt)                                                            \
    return dt == DT_F16 ? gemv_group_launch<DT_F16, mt, rt>(epi, g, block, lds, st)    \
                        : gemv_group_launch<DT_BF16, mt, rt>(epi, g, block, lds, st);
  SPEAR_GEMV_SHAPES(SPEAR_GEMV_GROUP_CASE)
#undef SPEAR_GEMV_GROUP_CASE
  return hipErrorInvalidValue;
}

hipError_t SPEAR_W(launch_gemm)(int dt, int epi, const GemmParams& p, hipStream_t st) {
  // split-K needs its partial tiles and tile counters (workspace); the
  // 256-token tile takes the plain and the semi-fused epilogue only
  const bool loc = epi == EPI_LOCAL || epi == EPI_LOCAL_I8;
  if (p.S < 1 || (p.S > 1 && (!p.ypart || !p.ctr || (loc && !p.epart))) ||
      (p.S != 1 && p.S != 2 && p.S != 4 && p.S != 8) ||
      (epi == EPI_LOCAL_I8 && (!p.A8 || !p.sa || !p.B8 || !p.sb)) ||
      (p.tmw != 2 && p.tmw != 4) || (p.tmw == 4 && loc))
    return hipErrorInvalidValue;
  const int TM = 64 * p.tmw;
  const int tm = (p.M + TM - 1) / TM, tn = (p.N + kGemmTN - 1) / kGemmTN;
  const unsigned grid = (unsigned)(tm * tn * p.S);
  if (grid == 0) return hipSuccess;
  size_t lds = (size_t)2 * (TM + kGemmTN) * kGemmLdsRow * 2;
  if (loc) lds += (size_t)2 * kGemmEcRows * kGemmLdsRow * 2;
#define SPEAR_GEMM_GO(E, W)                                                            \
  do {                                                                                 \
    hipError_t err = allow_lds(k_gemm<DTC, E, W, SPEAR_WB>, lds);                      \
    if (err != hipSuccess) return err;                                                 \
    hipLaunchKernelGGL((k_gemm<DTC, E, W, SPEAR_WB>), dim3(grid), dim3(128 * W), lds, st, p); \
  } while (0)
  if (p.roles == 2 || p.roles == 3) {
    // loading and multiplying waves: 256 x 128 (roles 2) or 256 x 256
    // (roles 3) tiles, one K-slice
    if (p.tmw != 4 || p.S != 1 || (epi != EPI_NONE && epi != EPI_READY)) return hipErrorInvalidValue;
    const int tnb = p.roles == 3 ? 2 : 1;
    const unsigned gws = (unsigned)(tm * ((p.N + 128 * tnb - 1) / (128 * tnb)));
    // unpadded activation stages, padded weight stages; the EC epilogue
    // reuses the space for v_hi, v_lo [256][72] and B [rows][72]
    const size_t lws = std::max((size_t)2 * TM * kGemmTK * 2 + (size_t)2 * 128 * tnb * kGemmLdsRow * 2,
                                (size_t)(2 * TM + 128 * tnb) * kGemmLdsRow * 2);
#define SPEAR_GEMM_WS(E, B)                                                               \
  do {                                                                                    \
    hipError_t err = allow_lds(k_gemm_ws<DTC, E, B, SPEAR_WB>, lws);                      \
    if (err != hipSuccess) return err;                                                    \
    hipLaunchKernelGGL((k_gemm_ws<DTC, E, B, SPEAR_WB>), dim3(gws), dim3(256 * (1 + B)), lws, st, p); \
  } while (0)
    SPEAR_DT_SWITCH(dt, {
      if (tnb == 2) {
        if (epi == EPI_NONE) SPEAR_GEMM_WS(EPI_NONE, 2);
        else SPEAR_GEMM_WS(EPI_READY, 2);
      } else {
        if (epi == EPI_NONE) SPEAR_GEMM_WS(EPI_NONE, 1);
        else SPEAR_GEMM_WS(EPI_READY, 1);
      }
    });
#undef SPEAR_GEMM_WS
    return hipGetLastError();
  }
  SPEAR_DT_SWITCH(dt, {
    if (p.tmw == 4) {
      if (epi == EPI_NONE) SPEAR_GEMM_GO(EPI_NONE, 4);
      else SPEAR_GEMM_GO(EPI_READY, 4);
    } else if (epi == EPI_NONE) {
      SPEAR_GEMM_GO(EPI_NONE, 2);
    } else if (epi == EPI_LOCAL) {
      SPEAR_GEMM_GO(EPI_LOCAL, 2);
    } else if (epi == EPI_LOCAL_I8) {
      SPEAR_GEMM_GO(EPI_LOCAL_I8, 2);
    } else {
      SPEAR_GEMM_GO(EPI_READY, 2);
    }
  });
#undef SPEAR_GEMM_GO
  return hipGetLastError();
}

}  // namespace spear
