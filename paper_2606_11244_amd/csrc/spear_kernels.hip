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
//   k_gemv     decode: split-K 4-bit product with MFMA, per-128 dequant
//              correction, cross-wave and cross-workgroup reduction, and an
//              epilogue adding B v; in the fused variant the same grid's first
//              workgroups run k_ec's work and publish v through a flag
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

// Last-arriver detection with an epoch-tagged 64-bit counter: the high word
// holds the call's epoch, the low word the arrivals of that epoch. A counter
// left over from another call (any other epoch) restarts at 1. Returns true
// for the arrival that completes `total`.
__device__ __forceinline__ bool arrive_last(unsigned long long* ctr, uint32_t epoch, uint32_t total) {
  unsigned long long old = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (;;) {
    const uint32_t e = (uint32_t)(old >> 32);
    const unsigned long long nv =
        (e == epoch) ? old + 1ull : (((unsigned long long)epoch << 32) | 1ull);
    if (__hip_atomic_compare_exchange_strong(ctr, &old, nv, __ATOMIC_ACQ_REL, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return (uint32_t)nv == total;
  }
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
// sum over the block's four waves in a fixed order.
// ---------------------------------------------------------------------------
template <int DT>
__device__ void ec_project_tile(const EcParams& e, int tb, int it_beg, int it_end, float* u_lds) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int m = tb * kTokTile + lr;
  const bool mval = m < e.M;
  const int RTe = (e.R1 + 15) >> 4;
  const uint16_t* xrow = e.x + (size_t)(mval ? m : 0) * e.K;
  for (int tg0 = 0; tg0 < RTe; tg0 += 4) {
    const int nt = min(4, RTe - tg0);
    f32x4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    const uint16_t* rsrc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = (tg0 + t) * 16 + lr;
      rsrc[t] = (t < nt && j < e.r) ? e.A + (size_t)j * e.K
                : (t < nt && j == e.r && e.gate == GATE_SIGMOID) ? e.wg
                                                                : nullptr;
    }
    for (int it = it_beg + wave; it < it_end; it += 4) {
      const int k = it * kIterK + 32 * lg;
      u32x4 xv[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        xv[jj] = mval ? ldg16(xrow + k + 8 * jj) : u32x4{0, 0, 0, 0};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        if (t < nt) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const u32x4 a = rsrc[t] ? ldg16(rsrc[t] + k + 8 * jj) : u32x4{0, 0, 0, 0};
            acc[t] = mfma16<DT>(a, xv[jj], acc[t]);
          }
        }
      }
    }
    // deterministic cross-wave sum: wave 0 stores, waves 1..3 add in order
    for (int w = 0; w < 4; ++w) {
      __syncthreads();
      if (wave == w) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
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
  const int tid = threadIdx.x;
  const int r = e.r;
  if (e.gate == GATE_TANH) {
    for (int t = 0; t < cnt; ++t) {
      const float* u = u_lds + t * e.R1p;
      for (int i = tid; i < e.h; i += 256) {
        float a = act2f<DT>(e.b1[i]);
        const uint16_t* w1 = e.W1 + (size_t)i * r;
        for (int j = 0; j < r; ++j) a += act2f<DT>(w1[j]) * u[j];
        hid[i] = a > 0.f ? a : 0.f;
      }
      __syncthreads();
      for (int j = tid; j < r; j += 256) {
        float a = act2f<DT>(e.b2[j]);
        const uint16_t* w2 = e.W2 + (size_t)j * e.h;
        for (int i = 0; i < e.h; ++i) a += act2f<DT>(w2[i]) * hid[i];
        v_tile[t * r + j] = e.alpha * (1.f + tanhf(a)) * u[j];
      }
      __syncthreads();
    }
  } else {
    for (int idx = tid; idx < cnt * r; idx += 256) {
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
// (last arriver), applies the gate and publishes v (fp32, and act-dtype
// hi/lo parts when requested), then releases flag[tb] if there is one.
template <int DT>
__device__ void ec_block(const EcParams& e, int tb, int p, char* smem) {
  __shared__ int s_last;
  const int tid = threadIdx.x;
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
    for (int idx = tid; idx < cnt * e.R1; idx += 256) {
      const int t = idx / e.R1, j = idx - t * e.R1;
      part[idx] = u_lds[t * e.R1p + j];
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = arrive_last(e.ctr + tb, e.epoch, (uint32_t)e.P) ? 1 : 0;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    const float* base = e.upart + (size_t)tb * e.P * kTokTile * e.R1;
    for (int idx = tid; idx < cnt * e.R1; idx += 256) {
      float a = 0.f;
      for (int q = 0; q < e.P; ++q) a += base[(size_t)q * kTokTile * e.R1 + idx];
      const int t = idx / e.R1, j = idx - t * e.R1;
      u_lds[t * e.R1p + j] = a;
    }
    __syncthreads();
  }

  if (e.raw) {
    for (int idx = tid; idx < cnt * e.R1; idx += 256) {
      const int t = idx / e.R1, j = idx - t * e.R1;
      e.u_out[(size_t)(m0 + t) * e.R1 + j] = u_lds[t * e.R1p + j];
    }
    return;
  }

  ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
  for (int idx = tid; idx < cnt * e.r; idx += 256)
    e.v[(size_t)m0 * e.r + idx] = v_tile[idx];
  if (e.vh) {
    for (int idx = tid; idx < cnt * e.vstride; idx += 256) {
      const int t = idx / e.vstride, j = idx - t * e.vstride;
      float val = j < e.r ? v_tile[t * e.r + j] : 0.f;
      const uint16_t hi = f2act<DT>(val);
      const uint16_t lo = f2act<DT>(val - act2f<DT>(hi));
      e.vh[(size_t)(m0 + t) * e.vstride + j] = hi;
      e.vl[(size_t)(m0 + t) * e.vstride + j] = lo;
    }
  }
  if (e.flag) {
    __threadfence();
    __syncthreads();
    if (tid == 0) __hip_atomic_store(e.flag + tb, e.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_ec(EcParams e) {
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
  for (int idx = threadIdx.x; idx < cnt * e.R1; idx += 256) {
    const int t = idx / e.R1, j = idx - t * e.R1;
    u_lds[t * e.R1p + j] = e.u_out[(size_t)(m0 + t) * e.R1 + j];
  }
  __syncthreads();
  ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
  for (int idx = threadIdx.x; idx < cnt * e.r; idx += 256) e.v[(size_t)m0 * e.r + idx] = v_tile[idx];
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

// ---------------------------------------------------------------------------
// Decode GEMV. Block = 4 waves on RT row tiles (16 rows each) and one K-slice;
// waves take the slice's 128-wide iterations round robin. Per iteration and
// row tile a lane loads 16 B of codes (32 codes of one row), the MFMA runs on
// biased codes (1024+q or 128+q, exact) against the matching activations,
// and the group's scale and zero are applied in fp32:
//   sum_k x (q - z) s = s * ( sum_k x (bias + q) - (bias + z) * sum_k x ),
// with sum_k x taken by an MFMA against ones.
// ---------------------------------------------------------------------------
template <int DT, int MT, int RT, int EPI>
__global__ __launch_bounds__(256) void k_gemv(GemvParams a) {
  extern __shared__ __attribute__((aligned(16))) char smem[];
  __shared__ int s_flag;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  int bid = blockIdx.x;
  if constexpr (EPI == EPI_FUSED) {
    if (bid < a.n_prod) {
      ec_block<DT>(a.ec, bid / a.ec.P, bid % a.ec.P, smem);
      return;
    }
    bid -= a.n_prod;
  }
  constexpr int RB = 16 * RT;
  const int rb = bid / a.S, s = bid - (bid / a.S) * a.S;
  const int n0 = rb * RB;
  const int M = a.M, N = a.N, K = a.K, G = a.G;
  const int IT = K / kIterK;
  const int it_beg = s * a.ips, it_end = min(IT, it_beg + a.ips);
  const int g_beg = (it_beg * kIterK) / G;
  const int g_end = (it_end * kIterK + G - 1) / G;
  const int ngs = max(1, g_end - g_beg);

  // stage this block's scales and zero points: [group][row]
  uint16_t* s_lds = (uint16_t*)smem;
  uint8_t* z_lds = (uint8_t*)(smem + align_up((size_t)ngs * RB * 2, 16));
  for (int idx = tid; idx < ngs * RB; idx += 256) {
    const int row = idx / ngs, gg = idx - row * ngs;
    const int n = n0 + row;
    const bool ok = n < N && (g_beg + gg) < a.ngroups;
    const size_t o = (size_t)n * a.ngroups + g_beg + gg;
    s_lds[gg * RB + row] = ok ? a.sc[o] : (uint16_t)0;
    z_lds[gg * RB + row] = ok ? a.zr[o] : (uint8_t)0;
  }
  __syncthreads();

  f32x4 acc[RT][MT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[t][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t kw = (size_t)(K >> 3);
  const uint32_t* wrow[RT];
  bool wval[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int n = n0 + 16 * t + lr;
    wval[t] = n < N;
    wrow[t] = a.qw + (size_t)(wval[t] ? n : 0) * kw + 4 * lg;
  }
  const uint16_t* xrow[MT];
  bool xval[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = 16 * mt + lr;
    xval[mt] = m < M;
    xrow[mt] = a.x + (size_t)(xval[mt] ? m : 0) * K + 32 * lg;
  }
  constexpr float kBias = code_bias<DT>();

  for (int it = it_beg + wave; it < it_end; it += 4) {
    const int k0 = it * kIterK;
    u32x4 wv[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) wv[t] = wval[t] ? ldg16(wrow[t] + (k0 >> 3)) : u32x4{0, 0, 0, 0};
    u32x4 xv[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        xv[mt][jj] = xval[mt] ? ldg16(xrow[mt] + k0 + 8 * jj) : u32x4{0, 0, 0, 0};
    f32x4 xb[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      xb[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) xb[mt] = mfma16<DT>(ones8<DT>(), xv[mt][jj], xb[mt]);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) xv[mt][jj] = pair_like_codes(xv[mt][jj]);
    }
    const int gg = k0 / G - g_beg;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
      const u32x2 s4 = *(const u32x2*)(s_lds + gg * RB + 16 * t + 4 * lg);
      const uint32_t z4 = *(const uint32_t*)(z_lds + gg * RB + 16 * t + 4 * lg);
      float sf[4], cf[4];
      sf[0] = h2f((uint16_t)(s4[0] & 0xFFFF));
      sf[1] = h2f((uint16_t)(s4[0] >> 16));
      sf[2] = h2f((uint16_t)(s4[1] & 0xFFFF));
      sf[3] = h2f((uint16_t)(s4[1] >> 16));
#pragma unroll
      for (int i = 0; i < 4; ++i) cf[i] = kBias + (float)((z4 >> (8 * i)) & 0xFF);
      u32x4 wd[4];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) wd[jj] = unpack_biased<DT>(wv[t][jj]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 pacc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) pacc = mfma16<DT>(wd[jj], xv[mt][jj], pacc);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[t][mt][i] += sf[i] * (pacc[i] - cf[i] * xb[mt][i]);
      }
    }
  }

  // cross-wave reduction (fixed order 0 + 1 + 2 + 3) into wave 0
  __syncthreads();
  float* red = (float*)smem;
  if (wave > 0) {
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        *(f32x4*)(red + (((wave - 1) * RT * MT + t * MT + mt) * 64 + lane) * 4) = acc[t][mt];
  }
  __syncthreads();
  float* yacc = (float*)(smem + gemv_lds_y_off(ngs, RT, MT));
  constexpr int YS = 16 * MT;  // row stride of yacc
  if (wave == 0) {
#pragma unroll
    for (int w = 1; w < 4; ++w)
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[t][mt] += *(const f32x4*)(red + (((w - 1) * RT * MT + t * MT + mt) * 64 + lane) * 4);
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) yacc[(16 * t + 4 * lg + i) * YS + 16 * mt + lr] = acc[t][mt][i];
  }
  __syncthreads();

  // cross-workgroup split-K reduction: last arriver of the row block sums the
  // S partials in slice order
  if (a.S > 1) {
    for (int idx = tid; idx < RB * M; idx += 256) {
      const int m = idx / RB, row = idx - m * RB;
      const int n = n0 + row;
      if (n < N) a.ypart[((size_t)s * M + m) * N + n] = yacc[row * YS + m];
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_flag = arrive_last(a.rb_ctr + rb, a.epoch, (uint32_t)a.S) ? 1 : 0;
    __syncthreads();
    if (!s_flag) return;
    __threadfence();
    for (int idx = tid; idx < RB * M; idx += 256) {
      const int m = idx / RB, row = idx - m * RB;
      const int n = n0 + row;
      if (n < N) {
        float t = 0.f;
        for (int q = 0; q < a.S; ++q) t += a.ypart[((size_t)q * M + m) * N + n];
        yacc[row * YS + m] = t;
      }
    }
    __syncthreads();
  }

  if constexpr (EPI == EPI_NONE) {
    for (int idx = tid; idx < RB * M; idx += 256) {
      const int m = idx / RB, row = idx - m * RB;
      const int n = n0 + row;
      if (n < N) a.y[(size_t)m * N + n] = f2act<DT>(yacc[row * YS + m]);
    }
    return;
  } else {
    const EcParams& e = a.ec;
    char* ec_smem = smem + gemv_lds_e_off(ngs, RT, MT);
    float* v_tile = (float*)(ec_smem + ec_lds_v_off(e.R1p, e.h));
    const int ntb = (M + kTokTile - 1) / kTokTile;
    bool have_v = true;
    if constexpr (EPI == EPI_FUSED) {
      // bounded wait for the EC workgroups; on time-out compute v here
      if (tid == 0) {
        int ok = 1;
        for (int tb = 0; tb < ntb && ok; ++tb) {
          int polls = 0;
          while (__hip_atomic_load(e.flag + tb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != e.epoch) {
            if (++polls > a.wait_polls) { ok = 0; break; }
            __builtin_amdgcn_s_sleep(8);
          }
        }
        s_flag = ok;
      }
      __syncthreads();
      __threadfence();
      have_v = s_flag != 0;
    }
    const int r = a.r;
    for (int tb = 0; tb < ntb; ++tb) {
      const int m0 = tb * kTokTile, cnt = min(kTokTile, M - m0);
      if (have_v) {
        for (int idx = tid; idx < cnt * r; idx += 256) v_tile[idx] = e.v[(size_t)m0 * r + idx];
        __syncthreads();
      } else {
        float* u_lds = (float*)(ec_smem + ec_lds_u_off());
        float* hid = (float*)(ec_smem + ec_lds_hid_off(e.R1p));
        ec_project_tile<DT>(e, tb, 0, IT, u_lds);
        ec_gate_tile<DT>(e, cnt, u_lds, hid, v_tile);
      }
      for (int idx = tid; idx < RB * cnt; idx += 256) {
        const int t = idx / RB, row = idx - t * RB;
        const int n = n0 + row;
        if (n < N) {
          float yv = yacc[row * YS + m0 + t];
          const uint16_t* br = a.B + (size_t)n * r;
          const float* vr = v_tile + t * r;
          for (int j = 0; j < r; ++j) yv += act2f<DT>(br[j]) * vr[j];
          a.y[(size_t)(m0 + t) * N + n] = f2act<DT>(yv);
        }
      }
      __syncthreads();
    }
  }
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

  // per-thread global load assignments
  int xr[4], xc[4];
  bool xv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    xr[i] = c >> 3;
    xc[i] = (c & 7) * 8;
    xv[i] = m0 + xr[i] < M;
  }
  const int wr = tid >> 1, wh = tid & 1;
  const int wn_row = n0 + wr;
  const bool wok = wn_row < N;
  const uint32_t* wsrc = a.qw + (size_t)(wok ? wn_row : 0) * (K >> 3) + 4 * wh;
  const size_t srow = (size_t)(wok ? wn_row : 0) * a.ngroups;

  u32x4 xreg[4];
  u32x4 wreg;
  float sreg;
  int zreg;
  auto gload = [&](int kt) {
    const int k0 = kt * kGemmTK;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      xreg[i] = xv[i] ? ldg16(a.x + (size_t)(m0 + xr[i]) * K + k0 + xc[i]) : u32x4{0, 0, 0, 0};
    wreg = wok ? ldg16(wsrc + (k0 >> 3)) : u32x4{0, 0, 0, 0};
    const int g = k0 / a.G;
    sreg = wok ? h2f(a.sc[srow + g]) : 0.f;
    zreg = wok ? (int)a.zr[srow + g] : 0;
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

hipError_t launch_ec(int dt, const EcParams& e, int ntb, size_t lds, hipStream_t st) {
  const unsigned grid = (unsigned)(ntb * e.P);
  if (grid == 0) return hipSuccess;
  SPEAR_DT_SWITCH(dt, {
    hipError_t err = allow_lds(k_ec<DTC>, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_ec<DTC>, dim3(grid), dim3(256), lds, st, e);
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
static hipError_t gemv_epi(int epi, const GemvParams& p, int grid, size_t lds, hipStream_t st) {
  hipError_t err = epi == EPI_NONE    ? allow_lds(k_gemv<DT, MT, RT, EPI_NONE>, lds)
                   : epi == EPI_READY ? allow_lds(k_gemv<DT, MT, RT, EPI_READY>, lds)
                                      : allow_lds(k_gemv<DT, MT, RT, EPI_FUSED>, lds);
  if (err != hipSuccess) return err;
  if (epi == EPI_NONE)
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_NONE>), dim3(grid), dim3(256), lds, st, p);
  else if (epi == EPI_READY)
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_READY>), dim3(grid), dim3(256), lds, st, p);
  else
    hipLaunchKernelGGL((k_gemv<DT, MT, RT, EPI_FUSED>), dim3(grid), dim3(256), lds, st, p);
  return hipGetLastError();
}

hipError_t launch_gemv(int dt, int MT, int RT, int epi, const GemvParams& p, int grid, size_t lds,
                       hipStream_t st) {
  if (grid == 0) return hipSuccess;
  // supported (MT, RT): (1,4) (2,2) (3,1) (4,1)
  SPEAR_DT_SWITCH(dt, {
    if (MT == 1 && RT == 4) return gemv_epi<DTC, 1, 4>(epi, p, grid, lds, st);
    if (MT == 2 && RT == 2) return gemv_epi<DTC, 2, 2>(epi, p, grid, lds, st);
    if (MT == 3 && RT == 1) return gemv_epi<DTC, 3, 1>(epi, p, grid, lds, st);
    if (MT == 4 && RT == 1) return gemv_epi<DTC, 4, 1>(epi, p, grid, lds, st);
  });
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
