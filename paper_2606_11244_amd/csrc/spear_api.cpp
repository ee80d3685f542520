// Host side of the C ABI (include/spear.h): argument validation, the
// phase-aware dispatch plan (SPEAR section 4.1), workspace layout and the
// launch sequence of each path. No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>

#include "../../include/spear.h"
#include "spear_internal.h"

using namespace spear;

namespace {

std::atomic<int32_t> g_wait_polls{1 << 16};
// tuning override of the GEMV shape (0 = automatic): row tiles per block,
// K-slices per row group, waves per block
std::atomic<int32_t> g_ov_rt{0}, g_ov_s{0}, g_ov_nw{0}, g_ov_gs{0}, g_ov_gt{0}, g_ov_nst{0}, g_ov_gr{0};

// Token counts at or below this run the 4-bit product as a split-K GEMV; above
// it the LDS-tiled MFMA GEMM. The same bound separates decode (fully fused
// EC) from prefill (semi-fused EC pre-kernel) under SPEAR_PATH_AUTO.
constexpr int64_t kGemvMaxM = 64;      // the GEMV kernels take up to this many tokens
constexpr int64_t kAutoGemvMaxM = 32;  // AUTO: GEMV kernels up to here, GEMM kernels above
constexpr int64_t kLocalMaxM = 32;   // local EC variant: at most two token tiles
constexpr size_t kLocalRestageMax = 24u << 20;  // local EC: A and w_g staged per call
// Largest staged slice of x in a GEMV block's LDS (16 tokens x 2048 K fit).
constexpr size_t kXLdsMax = 66 * 1024;
// Fused EC: the consumers gather the K-slices' partial sums themselves when
// there are at most this many words per launch (slices x tokens x (r + 1)).
constexpr int64_t kGatherMaxWords = 1024;
constexpr int kEcWaves = 8;  // waves of an EC pre-kernel block (decode)
constexpr size_t kMaxLds = 160 * 1024;  // LDS of one CU
// Fused EC: consumers poll the published data directly (instead of a ready
// counter) when it is at most this many words and the grid this small.
constexpr int64_t kDirectMaxWords = 512;
constexpr int kDirectMaxGrid = 512;

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Resolved {
  spear_plan_t plan;
  bool ec, gemv;
  int wb;  // weight code width: 4 or 3
  int dt, gate, G, ngroups, IT, r, R1, R1p, h, vstride;
  int MT, RT, NW, nrg, S, ips, iw;            // GEMV shape
  int nst;                                    // GEMV stages of codes in flight per wave
  int Sg;                                     // GEMM K-slices
  int gtmw;                                   // GEMM token waves (2: 128-token tiles, 4: 256)
  int groles;                                 // GEMM wave roles (1: every wave both, 2, 3: split)
  int ntb, P, eips, PG, tpg, ec_mode, ec_ipp, ec_block, n_prod;  // EC shape
  int xlds, xstride, bpre, lds_y, lds_e, lds_b, lds_g, lds_ev, lds_sz, lds_a;
  size_t off_vtag, off_upart, off_v, off_vh, off_vl, off_u, off_ypart, off_eupart, off_gpart,
      off_epart;
  size_t tag_bytes;  // fused path: bytes of its tagged region at off_vtag
  int npub, direct;
  size_t lds_gemv, lds_prod, lds_gate;
};

bool misaligned(const void* p) { return p && (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

spear_status_t validate_shape(const spear_problem_t* p, bool with_ec) {
  if (!p) return SPEAR_E_NULL;
  if (p->M < 0 || p->N < 0 || p->K <= 0 || p->K % kIterK) return SPEAR_E_SHAPE;
  if (p->act_dtype != SPEAR_F16 && p->act_dtype != SPEAR_BF16) return SPEAR_E_DTYPE;
  if (p->weight_bits != 0 && p->weight_bits != 4 && p->weight_bits != 3) return SPEAR_E_DTYPE;
  const int64_t G = (p->group_size == 0) ? p->K : p->group_size;
  if (G <= 0 || G % kIterK || p->K % G) return SPEAR_E_SHAPE;
  // every buffer stays below 2 GiB (element counts below 2^30), so that the
  // kernels' 32-bit byte offsets and buffer-resource bounds cover it
  const int64_t lim = (int64_t)1 << 30;
  if (p->M * p->K >= lim || p->N * p->K >= lim || p->M * p->N >= lim) return SPEAR_E_SHAPE;
  if (p->force_path < SPEAR_PATH_AUTO || p->force_path > SPEAR_PATH_OVERLAP_2K)
    return SPEAR_E_UNSUPPORTED;
  if (with_ec) {
    if (p->rank < 0 || p->rank > 256) return SPEAR_E_SHAPE;
    if (p->gate_kind < SPEAR_GATE_ONE || p->gate_kind > SPEAR_GATE_TANH_MLP) return SPEAR_E_UNSUPPORTED;
    if (p->gate_hidden < 0 || p->gate_hidden > 1024) return SPEAR_E_SHAPE;
  }
  return SPEAR_OK;
}

// Split-K of the decode GEMV: K-slices are added until about `waves` waves
// (4096: 16 per CU) cover the 256 CUs, keeping at least two iterations per
// wave so that the pipeline has something to overlap, and with cap_iw > 0 at
// most cap_iw iterations per wave. Returns the slice length in iterations.
// At a single token the 4-bit product alone and the producer-fused EC
// variant aim at 2048 waves: on the 70B-shaped 8192-row modules a second
// K-slice only adds the slices' reduction (4-bit q: 11.4 us unsplit against
// 15.1 us in two slices; fused q, rank 64: 18.3 against 23.9). At 16 tokens
// the 1B down module is faster split in four, so the rule stays at one token.
int gemv_ips(int IT, int nrg, int NW, int waves = 4096, int cap_iw = 0) {
  int S = (int)std::lround((double)waves / ((double)nrg * NW));
  if (cap_iw > 0) S = std::max(S, (int)cdiv(IT, NW * cap_iw));
  S = std::max(1, std::min(S, std::max(1, IT / (2 * NW))));
  if (g_ov_s.load() > 0) S = std::min((int)g_ov_s.load(), IT);
  return (int)cdiv(IT, S);
}

// Row tiles per GEMV block for MT token tiles. With one token tile (decode)
// the 4-bit product alone and the local EC variant take the fewest rows per
// block that keep the launch within one round of co-resident blocks (256
// blocks of 512 threads, one per CU): a decode block's time is mostly load
// latency, so more blocks with fewer rows each finish sooner, until a second
// round would wait for the first (measured on the 1B- and 70B-shaped
// modules); when no choice fits one round, two row tiles. The producer-fused
// EC variant at a single token (kRtFused1) takes one row tile on layers of
// 4096 rows or more when that fits one round, else two, with at most 16
// iterations per wave (measured, rank 32 and 64: 8B q 11.6 us against 13.3,
// 8B down 18.6 against 24.0; the 1024-row k modules are faster on two row
// tiles, the 28672-deep 70B down split in two). The other EC variants take
// two row tiles, and every variant with more token tiles two or one (the
// local variant keeps one for two token tiles: registers). rt_force > 0
// imposes a row-tile count (grouped calls).
enum { kRtW4 = 0, kRtLocal = 1, kRtOther = 2, kRtFused1 = 3 };
constexpr int64_t kGemvRound = 256;
constexpr int kFusedCapIw = 16;
// The producer-fused variant at a single token on layers narrower than this
// takes one row tile and one K-slice when each wave then has at most
// kFusedCapIw iterations: no split-K reduction after the stream (70B k,
// 1024 x 8192, rank 64: 12.2 us against 14.0 us on two row tiles in four
// K-slices).
constexpr int64_t kFusedNarrowN = 4096;
int gemv_rt(int MT, int kind, int64_t N, int IT, int NW, int rt_force, int waves) {
  if (g_ov_rt.load() > 0) return g_ov_rt.load();
  if (rt_force > 0) return rt_force;
  if (MT == 1 && kind == kRtFused1) {
    // (narrow layers: one row tile, over all of K when that keeps each wave
    // within the iteration cap, see kFusedNarrowN)
    if (N < kFusedNarrowN && IT <= NW * kFusedCapIw) return 1;
    const int nrg = (int)cdiv(N, 16);
    const int S = (int)cdiv(IT, gemv_ips(IT, nrg, NW, waves, kFusedCapIw));
    return N >= 4096 && (int64_t)nrg * S <= kGemvRound ? 1 : 2;
  }
  if (MT == 1 && kind != kRtOther) {
    for (int RT = 1; RT <= 4; RT *= 2) {
      const int nrg = (int)cdiv(N, 16 * RT);
      const int S = (int)cdiv(IT, gemv_ips(IT, nrg, NW, waves));
      if ((int64_t)nrg * S <= kGemvRound) return RT;
    }
    return 2;
  }
  return MT <= 2 && !(kind == kRtLocal && MT == 2) ? 2 : 1;
}

spear_status_t resolve(const spear_problem_t* p, bool with_ec, Resolved* R, int rt_force = 0) {
  spear_status_t st = validate_shape(p, with_ec);
  if (st != SPEAR_OK) return st;
  Resolved& z = *R;
  std::memset(&z, 0, sizeof(z));
  const int64_t M = p->M, N = p->N, K = p->K;
  z.dt = p->act_dtype;
  z.wb = p->weight_bits == 3 ? 3 : 4;
  z.G = (int)((p->group_size == 0) ? K : p->group_size);
  z.ngroups = (int)(K / z.G);
  z.IT = (int)(K / kIterK);
  z.r = with_ec ? p->rank : 0;
  z.ec = z.r > 0;
  z.gate = z.ec ? p->gate_kind : GATE_ONE;
  z.R1 = z.r + (z.gate == GATE_SIGMOID ? 1 : 0);
  z.R1p = (int)cdiv(std::max(z.R1, 1), 16) * 16;
  z.h = z.gate == GATE_TANH ? (p->gate_hidden > 0 ? p->gate_hidden : 4 * z.r) : 0;
  z.vstride = (int)cdiv(std::max(z.r, 1), 32) * 32;

  // path. The local variant of the fused kernel (the GEMV waves project x on
  // A and w_g themselves) applies to ranks up to 16 with an elementwise gate:
  // each workgroup then reads A once more from L2, which stays cheap while A
  // is one 16-row tile, and no workgroup waits for another.
  int path = p->force_path;
  bool local_ok = z.ec && z.r <= 16 && M <= kLocalMaxM;
  if (local_ok) {
    // the block's K-slice of A and w_g is staged in LDS
    const int MT = (int)cdiv(M, 16);
    const int nw = g_ov_nw.load() > 0 ? std::max(1, std::min(8, (int)g_ov_nw.load())) : 8;
    const int RT = gemv_rt(MT, kRtLocal, N, z.IT, nw, rt_force, 4096);
    const int ips = gemv_ips(z.IT, (int)cdiv(N, 16 * RT), nw);
    const size_t abytes = (size_t)17 * (ips * kIterK + 8) * 2;
    const size_t partials = (size_t)nw * (RT + kLocalTiles) * MT * 1024;
    // every row group stages all of A and w_g once: keep that L2 traffic
    // bounded (wide layers at two token tiles have many row groups)
    const size_t restaged = (size_t)cdiv(N, 16 * RT) * 17 * K * 2;
    local_ok = abytes <= kLocalALds && abytes + partials + 32768 <= kMaxLds &&
               restaged <= kLocalRestageMax;
  }
  // the fully fused GEMM: the projection rides on the GEMM's activation
  // tiles (one 16-row tile of A plus w_g), the gate and v B^T in its epilogue
  const bool mfma_ok = z.ec && z.r <= 16;
  if (z.ec && path == SPEAR_PATH_FUSED_MFMA && !mfma_ok) return SPEAR_E_UNSUPPORTED;
  if (path == SPEAR_PATH_FUSED_GEMV && M > kGemvMaxM) return SPEAR_E_UNSUPPORTED;
  if (z.ec && path == SPEAR_PATH_FUSED_LOCAL && !local_ok) return SPEAR_E_UNSUPPORTED;
  // prefill: the fully fused GEMM while its tile grid is small (at most
  // one 128 x 128 tile per CU, split over K): the separate projection
  // kernel's fixed cost then outweighs the projection the N-tiles repeat
  const bool few_tiles = cdiv(M, kGemmTM) * cdiv(N, kGemmTN) <= 256;
  // the 256-token GEMM tile applies (see the tile choice below): the
  // semi-fused pair on it beats the fully fused GEMM on 128-token tiles
  // (counting each 4096 of K beyond the first as another round of tiles):
  // when those tiles fill the 256 CUs, or, up to 512 tokens on layers of at
  // least 32M weights, when a quarter of them do and the halved weight
  // traffic pays for the emptier grid (70B q: 57 us against 70 us on
  // 128-token tiles at 256 tokens; 8B down: 58 against 71). Never at 128
  // tokens or fewer, where the 256-token tile only adds empty rows (70B gate
  // at 64 tokens: 107 us on 128-token tiles, 168 us on 256).
  const int64_t t256 = cdiv(M, 256) * cdiv(N, kGemmTN) * std::max<int64_t>(1, K / 4096);
  const bool big_tiles =
      M > 128 && (t256 >= 256 || (M <= 512 && N * K >= ((int64_t)1 << 25) && t256 >= 64));
  // decode beyond the local variant: the producer-fused GEMV, except a
  // single token on very deep layers, where its producers' share of K
  // outlasts the separate projection kernel (70B down, K = 28672, rank 64:
  // 40.2 us on the two-kernel path against 47.9 us fused; at 16 tokens, and
  // at K = 14336, the fused GEMV is faster).
  // Between 2 and 32 tokens on shallow layers (K <= 4096) the two-kernel
  // path wins too: the fused GEMV's EC wave waits for producers whose work
  // grows with the tokens (1B gate at 32 tokens: 21.3 us against 28.3 us;
  // 8B q at 8 tokens: 17.7 against 20.9; deeper layers keep the fused GEMV).
  const bool deep1 = (M == 1 && K >= 16384) || (M > 1 && K <= 4096);
  // a single token on narrow layers at least 8192 deep: the producer-fused
  // GEMV on one row tile over all of K beats the local variant, whose
  // workgroups each restage A for their K-slice (1B down, 2048 x 8192,
  // rank 16: 11.2 us against 13.3 us)
  const bool narrow_deep1 = M == 1 && N < kFusedNarrowN && K >= 8192 &&
                            K / kIterK <= (kGemvMaxThreads / 64 - 1) * kFusedCapIw;
  if (path == SPEAR_PATH_AUTO || !z.ec)
    path = M > kAutoGemvMaxM ? (mfma_ok && few_tiles && !big_tiles ? SPEAR_PATH_FUSED_MFMA
                                                                   : SPEAR_PATH_UNFUSED_2K)
           : local_ok && !narrow_deep1 ? SPEAR_PATH_FUSED_LOCAL
           : deep1           ? SPEAR_PATH_UNFUSED_2K
                             : SPEAR_PATH_FUSED_GEMV;
  if (!with_ec) {
    // the 4-bit product alone: the GEMV up to kAutoGemvMaxM tokens, the
    // GEMM above; force_path picks the kernel (GEMV paths: the GEMV, up to
    // kGemvMaxM tokens; GEMM paths: the GEMM)
    const int fp = p->force_path;
    const bool want_gemv = fp == SPEAR_PATH_FUSED_GEMV || fp == SPEAR_PATH_FUSED_LOCAL;
    const bool want_gemm = fp == SPEAR_PATH_FUSED_MFMA || fp == SPEAR_PATH_UNFUSED_2K ||
                           fp == SPEAR_PATH_UNFUSED_CHAIN || fp == SPEAR_PATH_OVERLAP_2K;
    if (want_gemv && M > kGemvMaxM) return SPEAR_E_UNSUPPORTED;
    path = want_gemv ? SPEAR_PATH_FUSED_GEMV
           : want_gemm ? SPEAR_PATH_UNFUSED_2K
           : M <= kAutoGemvMaxM ? SPEAR_PATH_FUSED_GEMV : SPEAR_PATH_UNFUSED_2K;
  }
  const bool fmfma = z.ec && path == SPEAR_PATH_FUSED_MFMA;
  // the GEMV for the GEMV paths, and under the 4-bit product of the
  // two-kernel and chain paths up to kAutoGemvMaxM tokens (the GEMM above)
  z.gemv = !with_ec ? path == SPEAR_PATH_FUSED_GEMV
           : path == SPEAR_PATH_FUSED_GEMV || path == SPEAR_PATH_FUSED_LOCAL ||
                 (!fmfma && M <= kAutoGemvMaxM);
  z.plan.path = path;

  if (M == 0 || N == 0) {
    z.plan.num_launches = 0;
    return SPEAR_OK;
  }
  const bool fused = z.ec && path == SPEAR_PATH_FUSED_GEMV;
  const bool local = z.ec && path == SPEAR_PATH_FUSED_LOCAL;

  // 4-bit product shape
  if (z.gemv) {
    // A block owns RT 16-row tiles and a K-slice; its NW waves each pipeline
    // a contiguous chunk of iw iterations (128 K each). K-slices are added
    // until about 4096 waves cover the 256 CUs, keeping at least two
    // iterations per wave so that the pipeline has something to overlap.
    z.MT = (int)cdiv(M, 16);
    z.NW = 8;
    const bool fused1 = fused && M == 1;
    // (the naive chain and the overlapped pair run the 4-bit product alone)
    const bool w4_kernel = !z.ec || path == SPEAR_PATH_UNFUSED_CHAIN || path == SPEAR_PATH_OVERLAP_2K;
    const int rt_kind = local                                           ? kRtLocal
                        : w4_kernel                                 ? kRtW4
                        : fused1                                    ? kRtFused1
                                                                    : kRtOther;
    // one token: the 4-bit product alone, the producer-fused and the
    // semi-fused GEMV aim at 2048 waves (70B down, semi-fused: 38.8 us in one
    // K-slice against 40.7 us in two). Four to sixteen tokens (one token
    // tile) on layers of at least 8192 rows and 8192 K: the 4-bit product
    // alone and the producer-fused GEMV aim at 2048 waves too, and from
    // eight tokens on, layers too wide for one round of two-row-tile blocks
    // take four row tiles, since every row group's blocks read the whole
    // token tile of x (70B shapes at 16 tokens, 4-bit only: q 26.4 -> 19.9
    // us, gate 68.9 -> 46.1, down 61.1 -> 52.5; fused: q 32.9 -> 26.0, gate
    // 70.7 -> 57.5, down 72.0 -> 61.9). Measured worse and left alone: two
    // tokens on 70B down (one K-slice no longer stages x in LDS: 38.6 against
    // 32.6 us) and the 8B shapes at eight tokens (gate 15.9 against 13.2,
    // down 18.3 against 16.0).
    const bool tile1 = z.MT == 1 && M >= 4 && N >= 8192 && K >= 8192 &&
                       (rt_kind == kRtW4 || (fused && rt_kind == kRtOther));
    // (the producer-fused GEMV from four tokens on: 70B gate at 4 tokens
    // 70.9 -> 48.8 us; the 4-bit product alone keeps two row tiles there,
    // 36.0 against 39.7 us)
    const bool wide1 = tile1 && (M >= 8 || (fused && M >= 4)) && rt_force == 0 &&
                       g_ov_rt.load() == 0 && cdiv(N, 32) > kGemvRound;
    const int waves =
        (M == 1 && (rt_kind == kRtW4 || rt_kind == kRtOther)) || fused1 || tile1 ? 2048 : 4096;
    // 17 to 32 tokens (two token tiles) on the same layers: four row tiles
    // (two for the 4-bit product alone on layers that fit one round of
    // two-row-tile blocks, K < 16384), K split in two from K = 16384 on and
    // unsplit below, and four-wave blocks for the 4-bit product alone (70B
    // shapes at 32 tokens, 4-bit only: q 42.3 -> 27.3 us, gate 112.2 ->
    // 64.4, down 96.8 -> 61.1; fused: q 56.7 -> 40.1, gate 120.1 -> 79.7,
    // down 126.7 -> 92.2)
    const bool tile2 = z.MT == 2 && N >= 8192 && K >= 8192 && rt_force == 0 &&
                       g_ov_rt.load() == 0 && g_ov_s.load() == 0 && g_ov_nw.load() == 0 &&
                       (rt_kind == kRtW4 || (fused && rt_kind == kRtOther));
    const int s_tile2 = K >= 16384 ? 2 : 1;
    {
      // the fused variant's GEMV waves: one wave of the block is the EC wave
      const int nw = g_ov_nw.load() > 0 ? std::max(1, std::min(8, (int)g_ov_nw.load()))
                                        : fused1 ? kGemvMaxThreads / 64 - 1 : 8;
      z.RT = tile2 ? (fused || cdiv(N, 32) > kGemvRound || K >= 16384 ? 4 : 2)
             : wide1 ? 4
                     : gemv_rt(z.MT, rt_kind, N, z.IT, nw, rt_force, waves);
    }
    if (!gemv_shape_supported(z.MT, z.RT)) return SPEAR_E_UNSUPPORTED;
    // the EC variants add the EC wave to the workgroup
    const int epi = w4_kernel                                 ? EPI_NONE
                    : path == SPEAR_PATH_FUSED_GEMV           ? EPI_FUSED
                    : local                                   ? EPI_LOCAL
                                                              : EPI_READY;
    const int max_nw = kGemvMaxThreads / 64 - (epi == EPI_READY || epi == EPI_FUSED ? 1 : 0);
    z.NW = std::min(z.NW, max_nw);
    // the 4-bit product alone at a single token on layers too wide for one
    // round of blocks: four-wave blocks, two rounds of which share a CU
    // (70B gate: 30.8 us against 33.7 us with eight waves)
    if (rt_kind == kRtW4 && M == 1 && rt_force == 0 && g_ov_rt.load() == 0) {
      const int nrg = (int)cdiv(N, 16 * z.RT);
      if ((int64_t)nrg * cdiv(z.IT, gemv_ips(z.IT, nrg, z.NW, waves)) > kGemvRound) z.NW = 4;
    }
    // and on the four-row-tile blocks of eight to sixteen tokens (70B gate at
    // 16 tokens: 46.1 us against 55.0 with eight waves), and at 17 to 32
    // tokens on the layers above
    if ((wide1 || tile2) && rt_kind == kRtW4) z.NW = 4;
    if (g_ov_nw.load() > 0) z.NW = std::max(1, std::min(max_nw, (int)g_ov_nw.load()));
    z.nrg = (int)cdiv(N, 16 * z.RT);
    z.ips = tile2 ? (int)cdiv(z.IT, s_tile2)
            : fused1 && N < kFusedNarrowN && z.RT == 1 && z.IT <= z.NW * kFusedCapIw &&
                    g_ov_s.load() == 0
                ? z.IT
                : gemv_ips(z.IT, z.nrg, z.NW, waves, fused1 ? kFusedCapIw : 0);
    z.S = (int)cdiv(z.IT, z.ips);
    z.iw = (int)cdiv(z.ips, z.NW);
    z.nst = 2;
    if (g_ov_nst.load() > 0) {
      // a deeper pipeline: one token tile, the 4-bit-only, fused and
      // semi-fused variants
      const int n = g_ov_nst.load();
      if ((n != 2 && n != 4) || (n != 2 && (z.MT != 1 || epi == EPI_LOCAL)))
        return SPEAR_E_UNSUPPORTED;
      z.nst = n;
    }

    z.plan.split_k = z.S;
    z.plan.tile_m = 16 * z.MT;
    z.plan.tile_n = 16 * z.RT;
  } else {
    // prefill GEMM tile: 256 tokens (eight waves, one workgroup per CU)
    // while those tiles fill the 256 CUs, counting each 4096 of K beyond the
    // first as another round of them (measured: 1B down at M = 2048), else
    // 128 (four waves, two workgroups per CU); the fully fused variant
    // takes 128
    z.gtmw = !fmfma && big_tiles ? 4 : 2;
    if (g_ov_gt.load() > 0) {
      z.gtmw = g_ov_gt.load() == 256 ? 4 : 2;
      if (fmfma && z.gtmw == 4) return SPEAR_E_UNSUPPORTED;
    }
    const int tm = 64 * z.gtmw;
    // K-slices (2, 4 or 8, each an even number of 64-wide steps, at least
    // four) while the tile grid alone fills less than the 256 CUs; the fully
    // fused variant splits its EC projection the same way
    const int64_t tiles = cdiv(M, tm) * cdiv(N, kGemmTN);
    const int steps = (int)(K / kGemmTK);
    z.Sg = 1;
    for (int S = 2; S <= 8; S *= 2)
      if (tiles * z.Sg < 256 && steps % (2 * S) == 0 && steps / S >= 4) z.Sg = S;
    if (g_ov_gs.load() > 0) {
      const int S = g_ov_gs.load();
      if (steps % (2 * S) != 0) return SPEAR_E_UNSUPPORTED;
      z.Sg = S;
    }
    // 256-token tiles in one K-slice (the plain and the semi-fused
    // epilogue): loading and multiplying waves (k_gemm_ws), on 256 x 256
    // tiles while those alone fill the 256 CUs, else 256 x 128
    const bool split_ok = z.gtmw == 4 && z.Sg == 1;
    z.groles = !split_ok ? 1 : cdiv(M, tm) * cdiv(N, 2 * kGemmTN) >= 256 ? 3 : 2;
    if (g_ov_gr.load() > 0) {
      z.groles = g_ov_gr.load();
      if (z.groles >= 2 && !split_ok) return SPEAR_E_UNSUPPORTED;
    }
    z.plan.split_k = z.Sg;
    z.plan.tile_m = tm;
    z.plan.tile_n = z.groles == 3 ? 2 * kGemmTN : kGemmTN;
  }

  // EC projection shape. Decode: one producer workgroup per (token tile,
  // K-slice, pair of 16-row tiles of [A; w_g]), each slice one pass of the
  // workgroup's waves, so that every producer is a single round of loads.
  // Prefill: one workgroup per token tile over all of K and all rows.
  z.ntb = (int)cdiv(M, kTokTile);
  if (fmfma) {
    z.P = 1;  // each GEMM workgroup projects its token tile over all of K
    z.PG = 1;
  } else if (local) {
    // the projection is split like the 4-bit product: one slice per K-slice
    z.P = z.S;
    z.PG = 1;
  } else if (z.ec) {
    const int RTe = (int)cdiv(z.R1, 16);
    if (z.gemv) {
      // fused producers are workgroups of the GEMV grid: its waves plus the EC wave
      const int nw = fused ? z.NW + 1 : kEcWaves;
      z.ec_block = 64 * nw;
      z.ec_ipp = 1;  // one iteration per wave: every producer is one round of loads
      z.eips = std::max(nw * z.ec_ipp, (int)cdiv(z.IT, 512 * nw));  // <= 512 * nw slices
      z.P = (int)cdiv(z.IT, z.eips);
      z.PG = (int)cdiv(RTe, kEcTiles);
      z.tpg = kEcTiles;
      z.ec_mode = path == SPEAR_PATH_UNFUSED_CHAIN ? EC_RAW : EC_LAST;
      if (fused && z.gate != GATE_TANH) {
        // gather mode when the slices' partials are few: with fewer, longer
        // slices if that keeps each producer within four passes
        const int64_t words = (int64_t)z.P * M * z.R1;
        const int64_t pmax = kGatherMaxWords / (M * z.R1);
        if (words <= kGatherMaxWords) {
          z.ec_mode = EC_GATHER;
        } else if (pmax >= 1 && cdiv(z.IT, pmax) <= 4 * nw * z.ec_ipp) {
          z.eips = (int)cdiv(z.IT, pmax);
          z.P = (int)cdiv(z.IT, z.eips);
          z.ec_mode = EC_GATHER;
        }
      }
      z.lds_prod = ec_block_lds(nw, z.R1p, z.h, z.r);
    } else {
      // eight-wave producers; while the token tiles alone leave CUs idle
      // (fewer than 256 workgroups), the rows of [A; w_g] are split into
      // groups of two 16-row tiles and K into slices (at least one pass of
      // one iteration per wave each), combined by the token tile's last
      // producer
      z.ec_block = 512;
      z.ec_ipp = 2;
      z.eips = z.IT;
      z.P = 1;
      z.PG = 1;
      z.tpg = RTe;
      if (z.ntb < 256 && z.ntb <= kMaxEcCounters) {
        z.PG = (int)cdiv(RTe, kEcTiles);
        z.tpg = kEcTiles;
        int P = 1;
        while ((int64_t)z.ntb * P * z.PG < 256 && cdiv(z.IT, 2 * P) >= 8) P *= 2;
        z.eips = (int)cdiv(z.IT, P);
        z.P = (int)cdiv(z.IT, z.eips);
        if (z.P > 1) z.ec_ipp = 1;
      }
      z.ec_mode = path == SPEAR_PATH_UNFUSED_CHAIN ? EC_RAW : EC_LAST;
      z.lds_prod = ec_block_lds(8, z.R1p, z.h, z.r);
    }
    z.lds_gate = ec_lds_bytes(z.R1p, z.h, z.r);
  }

  if (z.gemv) {
    // LDS of a GEMV block: [x slice | wave partials | gather scratch]
    // [yacc] [EC u/hidden/v] [rows of B] [scales and zero points]; the x
    // slice is staged only while the whole layout fits the CU's LDS
    const int RB = 16 * z.RT;
    z.xstride = z.ips * kIterK * 2 + 16;
    const size_t xbytes = (size_t)M * z.xstride;
    auto layout = [&](bool xl) {
      const int rtw = z.RT + (local ? kLocalTiles : 0);  // wave partial tiles
      size_t U = std::max((size_t)z.NW * rtw * z.MT * 1024, (size_t)z.S * 4);
      if (xl) U = std::max(U, xbytes);
      z.lds_y = (int)align_up(U, 16);
      z.lds_e = z.lds_y + z.RT * z.MT * 1024;
      z.lds_b = z.lds_g = z.lds_ev = z.lds_e;
      if (local) {
        // u [16 MT][R1p] and v [16 MT][r] (and the tanh-MLP gate's hidden
        // layer), the rows of B, the staged A, w_g
        const size_t hid = z.gate == GATE_TANH ? (size_t)local_tanh_cap((int)M, z.h) * z.h * 4 +
                                                     (size_t)tanh_stage_halves(z.h, z.r) * 2
                                               : 0;
        z.lds_b = (int)align_up(z.lds_e + (size_t)16 * z.MT * (z.R1p + z.r) * 4 + hid, 16);
        z.bpre = (z.r % 8) == 0 && RB * z.r / 8 <= 2 * 64 * z.NW;
        z.lds_a = (int)align_up(z.lds_b + (z.bpre ? (size_t)RB * z.r * 2 : 0), 16);
        z.lds_g = z.lds_ev = (int)(z.lds_a + (size_t)17 * (z.ips * kIterK + 8) * 2);
      } else if (z.ec) {
        z.lds_b = (int)(z.lds_e + ec_lds_bytes(z.R1p, z.h, z.r));
        z.bpre = (z.r % 8) == 0 && RB * z.r / 8 <= 2 * 64 * z.NW;
        z.lds_g = (int)align_up(z.lds_b + (z.bpre ? (size_t)RB * z.r * 2 : 0), 16);
        z.lds_ev = z.lds_g;
        if (fused && z.ec_mode == EC_GATHER)
          z.lds_ev = (int)(z.lds_g + (size_t)z.P * kTokTile * z.R1 * 4);
      }
      z.lds_sz = z.lds_ev + (z.ec && !local ? z.RT * z.MT * 1024 : 0);
      const int ipg = z.G / kIterK;
      const int ngb = (int)std::min<int64_t>(z.ngroups, cdiv(z.ips, ipg) + 1);
      z.lds_gemv = z.lds_sz + (size_t)RB * (ngb | 1) * 4;
    };
    z.xlds = xbytes <= kXLdsMax;
    layout(z.xlds);
    if (z.xlds && std::max(z.lds_gemv, z.lds_prod) > kMaxLds) {
      z.xlds = 0;
      layout(false);
    }
    if (std::max(z.lds_gemv, z.lds_prod) > kMaxLds) return local ? SPEAR_E_UNSUPPORTED : SPEAR_E_SHAPE;
  } else if (z.lds_prod > kMaxLds) {
    return SPEAR_E_SHAPE;
  }
  z.plan.ec_splits = z.ec ? z.P : 0;

  // launches and grid
  const int grid4 = z.gemv ? z.nrg * z.S : (int)(cdiv(M, z.plan.tile_m) * cdiv(N, z.plan.tile_n)) * z.Sg;
  if (!z.ec || local || fmfma) {
    z.plan.num_launches = 1;
    z.plan.grid = grid4;
  } else if (fused) {
    z.n_prod = z.ntb * z.P * z.PG;
    z.plan.num_launches = 1;
    z.plan.grid = z.n_prod + grid4;
  } else if (path == SPEAR_PATH_UNFUSED_2K) {
    z.plan.num_launches = 2;
    z.plan.grid = grid4;
  } else if (path == SPEAR_PATH_OVERLAP_2K) {
    z.plan.num_launches = 3;
    z.plan.grid = grid4;
  } else {  // chain
    z.plan.num_launches = 4;
    z.plan.grid = grid4;
  }

  // workspace layout. The first kCounterBytes hold every counter of every
  // kind of call at fixed offsets (the fused path's launch counters,
  // EC-slice counters, row-group counters); the split-K and EC-slice
  // counters return to zero after each call and the fused path's advance by
  // a whole launch step. Then comes the fused path's tagged region (no other
  // kind of call writes it), and every call's data regions start after it, so
  // any mix of calls can share one zero-initialised workspace and a tagged
  // word that is not this launch's carries an earlier launch's tag.
  size_t off = kDataBase;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  if (local) {
    if (z.S > 1) z.off_eupart = take((size_t)z.nrg * z.S * M * z.R1 * 4);
  } else if (fmfma) {
    // the slices' EC accumulators (split-K only)
    if (z.Sg > 1) z.off_epart = take((size_t)z.Sg * cdiv(M, kGemmTM) * cdiv(N, kGemmTN) * 16384);
  } else if (z.ec) {
    const bool partials = z.ec_mode != EC_GATHER && z.P * z.PG > 1;
    if (partials && z.ntb > kMaxEcCounters) return SPEAR_E_SHAPE;
    if (fused) {
      const size_t tag_bytes = (size_t)kVCopies * M * 8 *
                               (z.ec_mode == EC_GATHER ? (size_t)z.P * z.R1 : (size_t)z.r);
      if (tag_bytes > kTagBytes) return SPEAR_E_SHAPE;
      z.off_vtag = kCounterBytes;
      z.tag_bytes = tag_bytes;
      z.npub = z.ec_mode == EC_GATHER ? z.ntb * z.P * z.PG : z.ntb;
      // small problems: the consumers poll the tagged data itself rather
      // than the ready counter, saving the publishers' completion wait
      const int64_t words = z.ec_mode == EC_GATHER ? (int64_t)z.P * M * z.R1 : M * z.r;
      z.direct = words <= kDirectMaxWords && z.nrg * z.S <= kDirectMaxGrid;
    }
    if (partials) z.off_upart = take((size_t)z.ntb * z.P * kTokTile * z.R1 * 4);
    z.off_v = take((size_t)M * z.r * 4);
    if (!z.gemv && path == SPEAR_PATH_UNFUSED_2K) {
      z.off_vh = take((size_t)M * z.vstride * 2);
      z.off_vl = take((size_t)M * z.vstride * 2);
    }
    if (path == SPEAR_PATH_UNFUSED_CHAIN) z.off_u = take((size_t)M * z.R1 * 4);
  }
  if (z.gemv && z.S > 1) {
    if (z.nrg > kMaxRowCounters) return SPEAR_E_SHAPE;
    z.off_ypart = take((size_t)z.S * M * N * 4);
  }
  if (!z.gemv && z.Sg > 1) {
    const int64_t tiles = cdiv(M, z.plan.tile_m) * cdiv(N, kGemmTN);
    const size_t part = (size_t)z.Sg * tiles * z.plan.tile_m * kGemmTN * 4;
    // the kernel addresses the partial tiles with 32-bit offsets
    if (tiles > kMaxRowCounters || part >= ((size_t)1 << 31)) return SPEAR_E_SHAPE;
    z.off_gpart = take(part);
  }
  z.plan.workspace_bytes = off;
  return SPEAR_OK;
}

// Bytes of the packed codes of an [N][K] weight of this code width.
size_t code_bytes(const spear_problem_t* p) {
  return p->weight_bits == 3 ? (size_t)p->N * p->K / 8 * 3 : (size_t)p->N * p->K / 2;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

spear_status_t check_w4(const spear_problem_t* p, const void* x, const spear_w4_t* w, const void* y) {
  if (!w || !x || !y || !w->qweight || !w->scales || !w->zeros) return SPEAR_E_NULL;
  if (misaligned(x) || misaligned(y) || misaligned(w->qweight) || misaligned(w->scales) ||
      misaligned(w->zeros))
    return SPEAR_E_ALIGN;
  const size_t G = p->group_size == 0 ? (size_t)p->K : (size_t)p->group_size;
  const size_t ybytes = (size_t)p->M * p->N * 2;
  if (overlaps(y, ybytes, x, (size_t)p->M * p->K * 2) ||
      overlaps(y, ybytes, w->qweight, code_bytes(p)) ||
      overlaps(y, ybytes, w->scales, (size_t)p->N * (p->K / G) * 2) ||
      overlaps(y, ybytes, w->zeros, (size_t)p->N * (p->K / G)))
    return SPEAR_E_ALIAS;
  return SPEAR_OK;
}

spear_status_t check_ec(const spear_problem_t* p, const Resolved& z, const spear_ec_t* ec, const void* y) {
  if (!z.ec) return SPEAR_OK;
  if (!ec || !ec->A || !ec->B) return SPEAR_E_NULL;
  if (ec->ab_format != SPEAR_AB_ACT && ec->ab_format != SPEAR_AB_INT8) return SPEAR_E_DTYPE;
  const bool i8 = ec->ab_format == SPEAR_AB_INT8;
  if (i8 && (!ec->a_scale || !ec->b_scale)) return SPEAR_E_NULL;
  if (z.gate == GATE_SIGMOID && !ec->w_g) return SPEAR_E_NULL;
  if (z.gate == GATE_TANH && (!ec->W1 || !ec->b1 || !ec->W2 || !ec->b2)) return SPEAR_E_NULL;
  if (misaligned(ec->A) || misaligned(ec->B) || misaligned(ec->w_g) || misaligned(ec->W1) ||
      misaligned(ec->b1) || misaligned(ec->W2) || misaligned(ec->b2) ||
      (i8 && (misaligned(ec->a_scale) || misaligned(ec->b_scale))))
    return SPEAR_E_ALIGN;
  const size_t ybytes = (size_t)p->M * p->N * 2, eb = i8 ? 1 : 2;
  if (overlaps(y, ybytes, ec->A, (size_t)z.r * p->K * eb) ||
      overlaps(y, ybytes, ec->B, (size_t)p->N * z.r * eb) ||
      (i8 && (overlaps(y, ybytes, ec->a_scale, (size_t)z.r * 4) ||
              overlaps(y, ybytes, ec->b_scale, (size_t)p->N * 4))) ||
      (z.gate == GATE_SIGMOID && overlaps(y, ybytes, ec->w_g, (size_t)p->K * 2)))
    return SPEAR_E_ALIAS;
  return SPEAR_OK;
}

bool ab_int8(const spear_ec_t* ec) { return ec && ec->ab_format == SPEAR_AB_INT8; }

spear_status_t check_ws(const spear_problem_t* p, const Resolved& z, const void* y, void* ws,
                        size_t ws_bytes) {
  if (z.plan.workspace_bytes == 0) return SPEAR_OK;
  if (!ws || ws_bytes < z.plan.workspace_bytes) return SPEAR_E_WORKSPACE;
  if (misaligned(ws)) return SPEAR_E_ALIGN;
  if (overlaps(y, (size_t)p->M * p->N * 2, ws, z.plan.workspace_bytes)) return SPEAR_E_ALIAS;
  return SPEAR_OK;
}

EcParams make_ec(const spear_problem_t* p, const Resolved& z, const void* x, const spear_ec_t* ec,
                 char* ws) {
  EcParams e;
  std::memset(&e, 0, sizeof(e));
  e.x = (const uint16_t*)x;
  e.M = (int)p->M;
  e.K = (int)p->K;
  e.r = z.r;
  e.R1 = z.R1;
  e.R1p = z.R1p;
  e.h = z.h;
  e.gate = z.gate;
  e.P = z.P;
  e.ips = z.eips;
  e.PG = z.PG;
  e.tpg = z.tpg;
  e.mode = z.ec_mode;
  e.vstride = z.vstride;
  if (ec) {
    if (ab_int8(ec)) {
      e.A8 = (const int8_t*)ec->A;
      e.sa = ec->a_scale;
    } else {
      e.A = (const uint16_t*)ec->A;
    }
    e.wg = (const uint16_t*)ec->w_g;
    e.W1 = (const uint16_t*)ec->W1;
    e.b1 = (const uint16_t*)ec->b1;
    e.W2 = (const uint16_t*)ec->W2;
    e.b2 = (const uint16_t*)ec->b2;
    e.b_g = ec->b_g;
    e.alpha = ec->alpha;
  }
  if (ws) {
    e.ctr = (uint32_t*)(ws + kCtrEc);
    if (z.off_upart) e.upart = (float*)(ws + z.off_upart);
    e.v = (float*)(ws + z.off_v);
  }
  return e;
}

GemvParams make_gemv(const spear_problem_t* p, const Resolved& z, const void* x, const spear_w4_t* w,
                     void* y, const spear_ec_t* ec, char* ws) {
  GemvParams g;
  std::memset(&g, 0, sizeof(g));
  g.qw = w->qweight;
  g.sc = w->scales;
  g.zr = w->zeros;
  g.x = (const uint16_t*)x;
  g.y = (uint16_t*)y;
  g.M = (int)p->M;
  g.N = (int)p->N;
  g.K = (int)p->K;
  g.G = z.G;
  g.ngroups = z.ngroups;
  g.r = z.r;
  if (ab_int8(ec)) {
    g.B8 = (const int8_t*)ec->B;
    g.sb = ec->b_scale;
  } else {
    g.B = ec ? (const uint16_t*)ec->B : nullptr;
  }
  g.S = z.S;
  g.ips = z.ips;
  g.iw = z.iw;
  g.wait_polls = g_wait_polls.load();
  g.xlds = z.xlds;
  g.xstride = z.xstride;
  // B rows are staged in LDS as act dtype, or as INT8 codes and scales by
  // the local variant (the EC wave reads INT8 B from memory)
  g.bpre = ec && (!ab_int8(ec) || z.plan.path == SPEAR_PATH_FUSED_LOCAL) ? z.bpre : 0;
  g.lds_y = z.lds_y;
  g.lds_e = z.lds_e;
  g.lds_b = z.lds_b;
  g.lds_g = z.lds_g;
  g.lds_ev = z.lds_ev;
  g.lds_sz = z.lds_sz;
  g.lds_a = z.lds_a;
  if (ws && z.S > 1) {
    g.ypart = (float*)(ws + z.off_ypart);
    g.rb_ctr = (uint32_t*)(ws + kCtrRows);
  }
  return g;
}

GemmParams make_gemm(const spear_problem_t* p, const Resolved& z, const void* x, const spear_w4_t* w,
                     void* y, const spear_ec_t* ec, char* ws) {
  GemmParams g;
  std::memset(&g, 0, sizeof(g));
  g.S = std::max(1, z.Sg);
  g.tmw = z.gtmw ? z.gtmw : 2;
  g.roles = z.groles >= 2 ? z.groles : 1;
  if (ws && z.Sg > 1) {
    g.ypart = (float*)(ws + z.off_gpart);
    g.ctr = (uint32_t*)(ws + kCtrRows);
    if (z.off_epart) g.epart = (float*)(ws + z.off_epart);
  }
  g.qw = w->qweight;
  g.sc = w->scales;
  g.zr = w->zeros;
  g.x = (const uint16_t*)x;
  g.y = (uint16_t*)y;
  g.M = (int)p->M;
  g.N = (int)p->N;
  g.K = (int)p->K;
  g.G = z.G;
  g.ngroups = z.ngroups;
  g.r = z.r;
  g.vstride = z.vstride;
  const bool i8 = ab_int8(ec);
  if (ec && ws && z.off_vh) {
    if (i8) {
      g.B8 = (const int8_t*)ec->B;
      g.sb = ec->b_scale;
    } else {
      g.B = (const uint16_t*)ec->B;
    }
    g.vh = (const uint16_t*)(ws + z.off_vh);
    g.vl = (const uint16_t*)(ws + z.off_vl);
  }
  if (ec && z.plan.path == SPEAR_PATH_FUSED_MFMA) {
    if (i8) {
      g.A8 = (const int8_t*)ec->A;
      g.B8 = (const int8_t*)ec->B;
      g.sa = ec->a_scale;
      g.sb = ec->b_scale;
    } else {
      g.B = (const uint16_t*)ec->B;
      g.A = (const uint16_t*)ec->A;
    }
    g.wg = (const uint16_t*)ec->w_g;
    g.W1 = (const uint16_t*)ec->W1;
    g.b1 = (const uint16_t*)ec->b1;
    g.W2 = (const uint16_t*)ec->W2;
    g.b2 = (const uint16_t*)ec->b2;
    g.h = z.h;
    g.alpha = ec->alpha;
    g.b_g = ec->b_g;
    g.gate = z.gate;
  }
  return g;
}

spear_status_t hip_status(hipError_t e) { return e == hipSuccess ? SPEAR_OK : SPEAR_E_HIP; }

// The overlapped semi-fused path's side stream and fork/join events, one set
// per device, created on the first such call there and kept until the
// process ends. Default priority; non-blocking against the null stream.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;
SideStream g_side[64];

spear_status_t side_stream(SideStream** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return SPEAR_E_HIP;
  SideStream& ss = g_side[dev];
  if (!ss.s) {
    if (hipStreamCreateWithFlags(&ss.s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) != hipSuccess)
      return SPEAR_E_HIP;
  }
  *out = &ss;
  return SPEAR_OK;
}

// The kernels that read the packed codes, for the problem's code width.
hipError_t launch_gemv_wb(const Resolved& z, int epi, const GemvParams& p, int grid, int block,
                          size_t lds, hipStream_t st) {
  // the naive chain's 4-bit kernel and grouped launches keep two stages
  const int nst = epi == EPI_NONE || epi == EPI_READY || epi == EPI_FUSED ? z.nst : 2;
  return z.wb == 3 ? launch_gemv_w3(z.dt, z.MT, z.RT, epi, nst, p, grid, block, lds, st)
                   : launch_gemv_w4(z.dt, z.MT, z.RT, epi, nst, p, grid, block, lds, st);
}
hipError_t launch_gemm_wb(const Resolved& z, int epi, const GemmParams& p, hipStream_t st) {
  return z.wb == 3 ? launch_gemm_w3(z.dt, epi, p, st) : launch_gemm_w4(z.dt, epi, p, st);
}

// res: [M][N] act-dtype residual added before the output's single rounding, or null
spear_status_t run_w4(const spear_problem_t* p, const Resolved& z, const void* x, const spear_w4_t* w,
                      void* y, char* ws, hipStream_t st, const uint16_t* res = nullptr) {
  if (z.gemv) {
    GemvParams g = make_gemv(p, z, x, w, y, nullptr, ws);
    g.res = res;
    return hip_status(launch_gemv_wb(z, EPI_NONE, g, z.nrg * z.S, 64 * z.NW, z.lds_gemv, st));
  }
  GemmParams g = make_gemm(p, z, x, w, y, nullptr, ws);
  g.res = res;
  return hip_status(launch_gemm_wb(z, EPI_NONE, g, st));
}

// The layer on its planned path, after validation; res as in run_w4 (the
// chain adds it in its 4-bit kernel, every other path in its final store).
spear_status_t run_layer(const spear_problem_t* prob, const Resolved& z, const void* x,
                         const spear_w4_t* w, const spear_ec_t* ec, void* y, const uint16_t* res,
                         char* ws, hipStream_t s) {
  spear_status_t st = SPEAR_OK;
  if (!z.ec) return run_w4(prob, z, x, w, y, ws, s, res);

  EcParams e = make_ec(prob, z, x, ec, ws);
  const int path = z.plan.path;
  const int ec_grid = z.ntb * z.P * z.PG;
  if (path == SPEAR_PATH_FUSED_MFMA) {
    GemmParams g = make_gemm(prob, z, x, w, y, ec, ws);
    g.res = res;
    return hip_status(launch_gemm_wb(z, ab_int8(ec) ? EPI_LOCAL_I8 : EPI_LOCAL, g, s));
  }
  if (path == SPEAR_PATH_FUSED_LOCAL) {
    GemvParams g = make_gemv(prob, z, x, w, y, ec, ws);
    g.res = res;
    g.ec = e;
    if (z.S > 1) g.eupart = (float*)(ws + z.off_eupart);
    return hip_status(launch_gemv_wb(z, ab_int8(ec) ? EPI_LOCAL_I8 : EPI_LOCAL, g, z.nrg * z.S,
                                     64 * z.NW, z.lds_gemv, s));
  }
  if (path == SPEAR_PATH_FUSED_GEMV) {
    e.vtag = (unsigned long long*)(ws + z.off_vtag);
    e.gen = (unsigned long long*)(ws + kCtrGen);
    e.ready = (unsigned long long*)(ws + kCtrReady);
    e.npub = z.npub;
    e.direct = z.direct;
    e.v = nullptr;
    GemvParams g = make_gemv(prob, z, x, w, y, ec, ws);
    g.res = res;
    g.ec = e;
    g.n_prod = z.n_prod;
    g.grid_total = z.n_prod + z.nrg * z.S;
    const size_t lds = std::max(z.lds_gemv, z.lds_prod);
    return hip_status(launch_gemv_wb(z, EPI_FUSED, g, g.grid_total, 64 * (z.NW + 1), lds, s));
  }
  if (path == SPEAR_PATH_UNFUSED_2K) {
    if (!z.gemv) {
      e.vh = (uint16_t*)(ws + z.off_vh);
      e.vl = (uint16_t*)(ws + z.off_vl);
      e.v = nullptr;
    }
    st = hip_status(launch_ec(z.dt, e, ec_grid, z.ec_block, z.ec_ipp, z.lds_prod, s));
    if (st != SPEAR_OK) return st;
    if (z.gemv) {
      GemvParams g = make_gemv(prob, z, x, w, y, ec, ws);
      g.res = res;
      g.ec = e;
      return hip_status(launch_gemv_wb(z, EPI_READY, g, z.nrg * z.S, 64 * (z.NW + 1), z.lds_gemv,
                                       s));
    }
    GemmParams g = make_gemm(prob, z, x, w, y, ec, ws);
    g.res = res;
    return hip_status(launch_gemm_wb(z, EPI_READY, g, s));
  }
  if (path == SPEAR_PATH_OVERLAP_2K) {
    // fork: the EC pre-kernel (A x, gate, v in fp32) on the side stream,
    // after everything already on the caller's stream; the 4-bit product on
    // the caller's stream meanwhile; join before the final accumulation
    std::lock_guard<std::mutex> lk(g_side_mu);
    SideStream* ss = nullptr;
    if ((st = side_stream(&ss)) != SPEAR_OK) return st;
    if (hipEventRecord(ss->fork, s) != hipSuccess || hipStreamWaitEvent(ss->s, ss->fork, 0) != hipSuccess)
      return SPEAR_E_HIP;
    st = hip_status(launch_ec(z.dt, e, ec_grid, z.ec_block, z.ec_ipp, z.lds_prod, ss->s));
    if (st != SPEAR_OK) return st;
    if (hipEventRecord(ss->join, ss->s) != hipSuccess) return SPEAR_E_HIP;
    st = run_w4(prob, z, x, w, y, ws, s, res);
    if (st != SPEAR_OK) return st;
    if (hipStreamWaitEvent(s, ss->join, 0) != hipSuccess) return SPEAR_E_HIP;
    const bool i8o = ab_int8(ec);
    return hip_status(launch_ec_up_acc(z.dt, e.v, i8o ? nullptr : (const uint16_t*)ec->B,
                                       i8o ? (const int8_t*)ec->B : nullptr,
                                       i8o ? ec->b_scale : nullptr, (uint16_t*)y, (int)prob->M,
                                       (int)prob->N, z.r, s));
  }
  // naive chain: 4-bit product, projection, gate, reprojection + accumulate
  st = run_w4(prob, z, x, w, y, ws, s, res);
  if (st != SPEAR_OK) return st;
  e.u_out = (float*)(ws + z.off_u);
  st = hip_status(launch_ec(z.dt, e, ec_grid, z.ec_block, z.ec_ipp, z.lds_prod, s));
  if (st != SPEAR_OK) return st;
  st = hip_status(launch_gate(z.dt, e, z.ntb, z.lds_gate, s));
  if (st != SPEAR_OK) return st;
  const bool i8 = ab_int8(ec);
  return hip_status(launch_ec_up_acc(z.dt, e.v, i8 ? nullptr : (const uint16_t*)ec->B,
                                     i8 ? (const int8_t*)ec->B : nullptr, i8 ? ec->b_scale : nullptr,
                                     (uint16_t*)y, (int)prob->M, (int)prob->N, z.r, s));
}

// ---- grouped calls --------------------------------------------------------

size_t round256(size_t b) { return (b + 255) / 256 * 256; }

// y of one member against every buffer another member reads or writes
bool hits_member(const void* y, size_t yb, const spear_layer_call_t& c) {
  const spear_problem_t* p = c.prob;
  const size_t G = p->group_size == 0 ? (size_t)p->K : (size_t)p->group_size;
  if (overlaps(y, yb, c.x, (size_t)p->M * p->K * 2) || overlaps(y, yb, c.y, (size_t)p->M * p->N * 2) ||
      overlaps(y, yb, c.w->qweight, code_bytes(p)) ||
      overlaps(y, yb, c.w->scales, (size_t)p->N * (p->K / G) * 2) ||
      overlaps(y, yb, c.w->zeros, (size_t)p->N * (p->K / G)))
    return true;
  const spear_ec_t* ec = c.ec;
  if (!ec || p->rank == 0) return false;
  const size_t eb = ec->ab_format == SPEAR_AB_INT8 ? 1 : 2;
  const size_t r = (size_t)p->rank;
  const size_t h = p->gate_hidden > 0 ? (size_t)p->gate_hidden : 4 * r;
  return overlaps(y, yb, ec->A, r * p->K * eb) || overlaps(y, yb, ec->B, (size_t)p->N * r * eb) ||
         overlaps(y, yb, ec->a_scale, r * 4) || overlaps(y, yb, ec->b_scale, (size_t)p->N * 4) ||
         overlaps(y, yb, ec->w_g, (size_t)p->K * 2) || overlaps(y, yb, ec->W1, h * r * 2) ||
         overlaps(y, yb, ec->b1, h * 2) || overlaps(y, yb, ec->W2, r * h * 2) ||
         overlaps(y, yb, ec->b2, r * 2);
}

// The kernel variant a resolved member runs when it is a single GEMV launch
// without cross-launch state (the 4-bit product alone or the local EC
// variant); -1 otherwise.
int group_epi(const Resolved& z, const spear_ec_t* ec) {
  if (!z.gemv) return -1;
  if (!z.ec) return EPI_NONE;
  if (z.plan.path == SPEAR_PATH_FUSED_LOCAL) return ab_int8(ec) ? EPI_LOCAL_I8 : EPI_LOCAL;
  return -1;
}

// Group workspace: the counter block and the tagged region of every
// workspace, then each member's data region (its plan's bytes past
// kDataBase) in array order. A member run on its own takes the workspace as
// it is (its data regions start at kDataBase); in the one-launch case member
// i's data start after the earlier members' and its split-K counters follow
// theirs in the counter block. Either way the counter block and the tagged
// region keep their places, so the workspace may be shared with single calls.
spear_status_t group_resolve(int32_t n, const spear_layer_call_t* calls, Resolved* z,
                             size_t* data_off, size_t* total) {
  if (!calls || !total) return SPEAR_E_NULL;
  if (n < 1 || n > SPEAR_GROUP_MAX) return SPEAR_E_SHAPE;
  size_t sum = 0;
  bool any = false;
  for (int i = 0; i < n; ++i) {
    if (!calls[i].prob) return SPEAR_E_NULL;
    const spear_status_t st = resolve(calls[i].prob, calls[i].ec != nullptr, &z[i]);
    if (st != SPEAR_OK) return st;
    const size_t b = z[i].plan.workspace_bytes;
    if (b > 0 && b < kDataBase) return SPEAR_E_SHAPE;  // every layout starts with the counters
    any = any || b > 0;
    data_off[i] = sum;
    sum += round256(b > 0 ? b - kDataBase : 0);
  }
  *total = any ? kDataBase + sum : 0;
  return SPEAR_OK;
}

// ---- the library's own scratch (spear_w4ec_linear_noalloc) ---------------
// One array per GPU, allocated by the loader with the code object and
// zero-filled there, so that its counter block starts at zero without any
// call of ours clearing it. Its device address comes from
// hipGetSymbolAddress, once per device, with that device current: in host
// code the array's name is only a host-side stand-in, never passed to a
// kernel or a copy.
static __device__ __align__(256) unsigned char scratch[SPEAR_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// This device's copy of the scratch array (looked up on the first call on
// the device), or null with *err set.
void* device_scratch(spear_status_t* err) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *err = SPEAR_E_HIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *err = SPEAR_E_HIP;
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

spear_status_t spear_dispatch_plan(const spear_problem_t* prob, int32_t with_ec, spear_plan_t* out) {
  if (!prob || !out) return SPEAR_E_NULL;
  Resolved z;
  spear_status_t st = resolve(prob, with_ec != 0, &z);
  if (st != SPEAR_OK) return st;
  *out = z.plan;
  return SPEAR_OK;
}

spear_status_t spear_w4_linear(const spear_problem_t* prob, const void* x, const spear_w4_t* w,
                               void* y, void* workspace, size_t workspace_bytes, void* hip_stream) {
  Resolved z;
  spear_status_t st = resolve(prob, false, &z);
  if (st != SPEAR_OK) return st;
  if (prob->M == 0 || prob->N == 0) return SPEAR_OK;
  if ((st = check_w4(prob, x, w, y)) != SPEAR_OK) return st;
  if ((st = check_ws(prob, z, y, workspace, workspace_bytes)) != SPEAR_OK) return st;
  return run_w4(prob, z, x, w, y, (char*)workspace, (hipStream_t)hip_stream);
}

spear_status_t spear_w4ec_linear(const spear_problem_t* prob, const void* x, const spear_w4_t* w,
                                 const spear_ec_t* ec, void* y, void* workspace,
                                 size_t workspace_bytes, void* hip_stream) {
  Resolved z;
  spear_status_t st = resolve(prob, true, &z);
  if (st != SPEAR_OK) return st;
  if (prob->M == 0 || prob->N == 0) return SPEAR_OK;
  if ((st = check_w4(prob, x, w, y)) != SPEAR_OK) return st;
  if ((st = check_ec(prob, z, ec, y)) != SPEAR_OK) return st;
  if ((st = check_ws(prob, z, y, workspace, workspace_bytes)) != SPEAR_OK) return st;
  return run_layer(prob, z, x, w, ec, y, nullptr, (char*)workspace, (hipStream_t)hip_stream);
}

spear_status_t spear_w4ec_linear_noalloc(const spear_problem_t* prob, const void* x,
                                         const spear_w4_t* w, const spear_ec_t* ec, void* y,
                                         void* hip_stream) {
  Resolved z;
  spear_status_t st = resolve(prob, true, &z);
  if (st != SPEAR_OK) return st;
  if (prob->M == 0 || prob->N == 0) return SPEAR_OK;
  if (z.plan.workspace_bytes > SPEAR_SCRATCH_BYTES) return SPEAR_E_WORKSPACE;
  if ((st = check_w4(prob, x, w, y)) != SPEAR_OK) return st;
  if ((st = check_ec(prob, z, ec, y)) != SPEAR_OK) return st;
  void* ws = device_scratch(&st);
  if (!ws) return st;
  return run_layer(prob, z, x, w, ec, y, nullptr, (char*)ws, (hipStream_t)hip_stream);
}

spear_status_t spear_w4ec_linear_tail(const spear_problem_t* prob, const void* x,
                                      const spear_w4_t* w, const spear_ec_t* ec,
                                      const spear_tail_t* tail, void* y, void* workspace,
                                      size_t workspace_bytes, void* hip_stream) {
  Resolved z;
  spear_status_t st = resolve(prob, ec != nullptr, &z);
  if (st != SPEAR_OK) return st;
  if (!tail) return SPEAR_E_NULL;
  if (!std::isfinite(tail->eps) || tail->eps < 0.f) return SPEAR_E_SHAPE;
  if (prob->M == 0 || prob->N == 0) return SPEAR_OK;
  if ((st = check_w4(prob, x, w, y)) != SPEAR_OK) return st;
  if (ec && (st = check_ec(prob, z, ec, y)) != SPEAR_OK) return st;
  if (tail->norm_w && !tail->y_norm) return SPEAR_E_NULL;
  if (misaligned(tail->residual) || misaligned(tail->norm_w) || misaligned(tail->y_norm))
    return SPEAR_E_ALIGN;
  const size_t yb = (size_t)prob->M * prob->N * 2;
  const size_t xb = (size_t)prob->M * prob->K * 2;
  if (tail->residual && tail->residual != y && overlaps(tail->residual, yb, y, yb))
    return SPEAR_E_ALIAS;
  if (tail->norm_w &&
      (overlaps(tail->y_norm, yb, y, yb) || overlaps(tail->y_norm, yb, x, xb) ||
       overlaps(tail->y_norm, yb, tail->residual, yb) ||
       overlaps(tail->y_norm, yb, tail->norm_w, (size_t)prob->N * 2) ||
       overlaps(tail->y_norm, yb, workspace, z.plan.workspace_bytes)))
    return SPEAR_E_ALIAS;
  if ((st = check_ws(prob, z, y, workspace, workspace_bytes)) != SPEAR_OK) return st;
  hipStream_t s = (hipStream_t)hip_stream;
  st = run_layer(prob, z, x, w, ec, y, (const uint16_t*)tail->residual, (char*)workspace, s);
  if (st != SPEAR_OK || !tail->norm_w) return st;
  return hip_status(launch_rmsnorm(z.dt, (const uint16_t*)y, (const uint16_t*)tail->norm_w,
                                   tail->eps, (uint16_t*)tail->y_norm, (int)prob->M,
                                   (int)prob->N, s));
}

// The members of a grouped call that share one launch: those that run one
// single-launch GEMV variant (same variant, dtype, code width and token
// tiles), the largest such set of at least two members. in[i] marks them
// (their plans in z re-planned to one tiling where needed); returns their
// count (0: every member runs on its own), with the launch's variant in
// *epi_out and its first member in *first_out.
int group_select(int32_t n, const spear_layer_call_t* calls, Resolved* z, bool* in, int* epi_out,
                 int* first_out) {
  int key[SPEAR_GROUP_MAX];
  for (int i = 0; i < n; ++i) {
    const bool live = calls[i].prob->M > 0 && calls[i].prob->N > 0;
    const int epi_i = live ? group_epi(z[i], calls[i].ec) : -1;
    key[i] = epi_i < 0 ? -1 : ((epi_i * 2 + z[i].dt) * 8 + z[i].wb) * 64 + z[i].MT;
  }
  for (int i = 0; i < n; ++i) in[i] = false;
  int best = -1, best_cnt = 1;
  for (int i = 0; i < n; ++i) {
    if (key[i] < 0) continue;
    int cnt = 0;
    for (int j = 0; j < n; ++j) cnt += key[j] == key[i];
    if (cnt > best_cnt) best = key[i], best_cnt = cnt;
  }
  for (int i = 0; i < n; ++i) in[i] = best >= 0 && key[i] == best;
  int first = -1;
  for (int i = 0; i < n && first < 0; ++i)
    if (in[i]) first = i;
  const int epi = first >= 0 ? group_epi(z[first], calls[first].ec) : -1;
  // One launch needs one row-tile count and one wave count. Members that
  // differ are re-planned to a common row-tile count when that changes
  // nothing but the row tiling (same K-slices, iterations per wave and
  // waves, so the same sums in the same order); the largest such count
  // (fewest workgroups) wins. Without one, the set keeps the members that
  // share the first member's tiling.
  if (first >= 0) {
    bool same = true;
    for (int i = 0; i < n; ++i)
      if (in[i]) same = same && z[i].RT == z[first].RT && z[i].NW == z[first].NW;
    if (!same) {
      Resolved zz[SPEAR_GROUP_MAX];
      bool found = false;
      for (int rt = 4; rt >= 1 && !found; rt /= 2) {
        bool ok = true;
        for (int i = 0; i < n && ok; ++i) {
          if (!in[i]) continue;
          ok = resolve(calls[i].prob, calls[i].ec != nullptr, &zz[i], rt) == SPEAR_OK &&
               group_epi(zz[i], calls[i].ec) == epi && zz[i].RT == rt && zz[i].S == z[i].S &&
               zz[i].ips == z[i].ips && zz[i].iw == z[i].iw && zz[i].NW == z[i].NW &&
               zz[i].NW == z[first].NW &&
               zz[i].plan.workspace_bytes <= z[i].plan.workspace_bytes;
        }
        if (ok) {
          found = true;
          for (int i = 0; i < n; ++i)
            if (in[i]) z[i] = zz[i];
        }
      }
      if (!found)
        for (int i = 0; i < n; ++i)
          if (in[i]) in[i] = z[i].RT == z[first].RT && z[i].NW == z[first].NW;
    }
  }
  int n_in = 0, ctrs = 0;
  for (int i = 0; i < n; ++i)
    if (in[i]) {
      ++n_in;
      if (z[i].S > 1) ctrs += z[i].nrg;
    }
  if (n_in < 2 || ctrs > kMaxRowCounters) {
    for (int i = 0; i < n; ++i) in[i] = false;
    n_in = 0;
  }
  *epi_out = epi;
  *first_out = first;
  return n_in;
}

spear_status_t spear_group_workspace(int32_t n, const spear_layer_call_t* calls, size_t* out_bytes) {
  Resolved z[SPEAR_GROUP_MAX];
  size_t off[SPEAR_GROUP_MAX];
  return group_resolve(n, calls, z, off, out_bytes);
}

spear_status_t spear_group_launches(int32_t n, const spear_layer_call_t* calls, int32_t* out_launches) {
  if (!out_launches) return SPEAR_E_NULL;
  Resolved z[SPEAR_GROUP_MAX];
  size_t off[SPEAR_GROUP_MAX], total = 0;
  const spear_status_t st = group_resolve(n, calls, z, off, &total);
  if (st != SPEAR_OK) return st;
  bool in[SPEAR_GROUP_MAX];
  int epi = -1, first = -1;
  const int n_in = group_select(n, calls, z, in, &epi, &first);
  int32_t launches = n_in > 0 ? 1 : 0;
  for (int i = 0; i < n; ++i)
    if (!in[i] && calls[i].prob->M > 0 && calls[i].prob->N > 0) launches += z[i].plan.num_launches;
  *out_launches = launches;
  return SPEAR_OK;
}

spear_status_t spear_w4ec_linear_group(int32_t n, const spear_layer_call_t* calls, void* workspace,
                                       size_t workspace_bytes, void* hip_stream) {
  Resolved z[SPEAR_GROUP_MAX];
  size_t off[SPEAR_GROUP_MAX], total = 0;
  spear_status_t st = group_resolve(n, calls, z, off, &total);
  if (st != SPEAR_OK) return st;
  if (total > 0) {
    if (!workspace || workspace_bytes < total) return SPEAR_E_WORKSPACE;
    if (misaligned(workspace)) return SPEAR_E_ALIGN;
  }
  char* ws = (char*)workspace;
  // every member's own checks first: the cross-member checks below read the
  // other members' pointers
  for (int i = 0; i < n; ++i) {
    const spear_layer_call_t& c = calls[i];
    const spear_problem_t* p = c.prob;
    if (p->M == 0 || p->N == 0) continue;
    if ((st = check_w4(p, c.x, c.w, c.y)) != SPEAR_OK) return st;
    if (c.ec && (st = check_ec(p, z[i], c.ec, c.y)) != SPEAR_OK) return st;
  }
  for (int i = 0; i < n; ++i) {
    const spear_layer_call_t& c = calls[i];
    const spear_problem_t* p = c.prob;
    if (p->M == 0 || p->N == 0) continue;
    const size_t yb = (size_t)p->M * p->N * 2;
    if (overlaps(c.y, yb, workspace, total)) return SPEAR_E_ALIAS;
    for (int j = 0; j < n; ++j)
      if (j != i && calls[j].prob->M > 0 && calls[j].prob->N > 0 && hits_member(c.y, yb, calls[j]))
        return SPEAR_E_ALIAS;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  // Members of one single-launch GEMV variant share one launch; the other
  // members run one after another on the same stream, as their own calls
  // would. Every member's output is the one its own call writes.
  bool in[SPEAR_GROUP_MAX];
  int epi = -1, first = -1;
  const int n_in = group_select(n, calls, z, in, &epi, &first);
  for (int i = 0; i < n; ++i) {
    const spear_layer_call_t& c = calls[i];
    if (in[i] || c.prob->M == 0 || c.prob->N == 0) continue;
    st = run_layer(c.prob, z[i], c.x, c.w, c.ec, c.y, nullptr, ws, s);
    if (st != SPEAR_OK) return st;
  }
  if (n_in == 0) return SPEAR_OK;
  // local EC members whose blocks exceed one round together take four row
  // tiles each when that changes nothing but the row tiling (same K-slices,
  // iterations per wave and waves, so the same sums in the same order): the
  // staged A limits the local variant to one block per CU
  if ((epi == EPI_LOCAL || epi == EPI_LOCAL_I8) && z[first].MT == 1) {
    int64_t blocks = 0;
    for (int i = 0; i < n; ++i)
      if (in[i]) blocks += (int64_t)z[i].nrg * z[i].S;
    if (blocks > kGemvRound) {
      Resolved zz[SPEAR_GROUP_MAX];
      bool same = true;
      int64_t blocks4 = 0;
      for (int i = 0; i < n && same; ++i) {
        if (!in[i]) continue;
        same = resolve(calls[i].prob, true, &zz[i], 4) == SPEAR_OK &&
               group_epi(zz[i], calls[i].ec) == epi && zz[i].RT == 4 && zz[i].S == z[i].S &&
               zz[i].ips == z[i].ips && zz[i].iw == z[i].iw && zz[i].NW == z[i].NW &&
               zz[i].plan.workspace_bytes <= z[i].plan.workspace_bytes;
        blocks4 += (int64_t)zz[i].nrg * zz[i].S;
      }
      if (same && blocks4 < blocks)
        for (int i = 0; i < n; ++i)
          if (in[i]) z[i] = zz[i];
    }
  }
  // the launch's members, in array order, as GemvGroup slots
  GemvGroup g;
  std::memset(&g, 0, sizeof(g));
  size_t lds = 0;
  int ctr = 0, k = 0;
  for (int i = 0; i < n; ++i) {
    if (!in[i]) continue;
    const spear_layer_call_t& c = calls[i];
    // member i's data regions (offsets past the counter block) land in its
    // own slice; its row counters are placed explicitly
    char* wsi = ws ? ws + off[i] : nullptr;
    g.start[k + 1] = g.start[k] + z[i].nrg * z[i].S;
    GemvParams& q = g.p[k];
    q = make_gemv(c.prob, z[i], c.x, c.w, c.y, z[i].ec ? c.ec : nullptr, wsi);
    if (z[i].ec) {
      q.ec = make_ec(c.prob, z[i], c.x, c.ec, wsi);
      if (z[i].S > 1) q.eupart = (float*)(wsi + z[i].off_eupart);
    }
    if (z[i].S > 1) {
      q.rb_ctr = (uint32_t*)(ws + kCtrRows) + ctr;
      ctr += z[i].nrg;
    }
    lds = std::max(lds, z[i].lds_gemv);
    ++k;
  }
  g.n = k;
  const Resolved& z0 = z[first];
  return hip_status(z0.wb == 3
                        ? launch_gemv_group_w3(z0.dt, z0.MT, z0.RT, epi, g, 64 * z0.NW, lds, s)
                        : launch_gemv_group_w4(z0.dt, z0.MT, z0.RT, epi, g, 64 * z0.NW, lds, s));
}

spear_status_t spear_w4_dequant(const spear_problem_t* prob, const spear_w4_t* w, void* w_out,
                                void* hip_stream) {
  if (!prob || !w) return SPEAR_E_NULL;
  spear_problem_t q = *prob;
  q.M = 0;
  q.force_path = SPEAR_PATH_AUTO;
  spear_status_t st = validate_shape(&q, false);
  if (st != SPEAR_OK) return st;
  if (prob->N == 0) return SPEAR_OK;
  if (!w_out || !w->qweight || !w->scales || !w->zeros) return SPEAR_E_NULL;
  if (misaligned(w_out) || misaligned(w->qweight) || misaligned(w->scales) || misaligned(w->zeros))
    return SPEAR_E_ALIGN;
  const int G = (int)(prob->group_size == 0 ? prob->K : prob->group_size);
  const size_t outb = (size_t)prob->N * prob->K * 2;
  if (overlaps(w_out, outb, w->qweight, code_bytes(prob)) ||
      overlaps(w_out, outb, w->scales, (size_t)prob->N * (prob->K / G) * 2) ||
      overlaps(w_out, outb, w->zeros, (size_t)prob->N * (prob->K / G)))
    return SPEAR_E_ALIAS;
  const auto dq = prob->weight_bits == 3 ? launch_dequant_w3 : launch_dequant_w4;
  return hip_status(dq(prob->act_dtype, w->qweight, w->scales, w->zeros, (uint16_t*)w_out,
                       (int)prob->N, (int)prob->K, G, (hipStream_t)hip_stream));
}

spear_status_t spear_workspace_regions(const spear_problem_t* prob, int32_t with_ec,
                                       size_t* tag_begin, size_t* tag_end, size_t* data_begin,
                                       size_t* data_end) {
  if (!prob || !tag_begin || !tag_end || !data_begin || !data_end) return SPEAR_E_NULL;
  Resolved z;
  const spear_status_t st = resolve(prob, with_ec != 0, &z);
  if (st != SPEAR_OK) return st;
  *tag_begin = z.tag_bytes ? z.off_vtag : 0;
  *tag_end = z.tag_bytes ? z.off_vtag + z.tag_bytes : 0;
  const size_t ws = z.plan.workspace_bytes;
  *data_begin = ws > kDataBase ? kDataBase : 0;
  *data_end = ws > kDataBase ? ws : 0;
  return SPEAR_OK;
}

int32_t spear_set_wait_polls(int32_t polls) { return g_wait_polls.exchange(polls < 0 ? 0 : polls); }

void spear_set_gemv_shape(int32_t row_tiles, int32_t k_slices, int32_t waves) {
  g_ov_rt = row_tiles > 0 ? row_tiles : 0;
  g_ov_s = k_slices > 0 ? k_slices : 0;
  g_ov_nw = waves > 0 ? waves : 0;
}

void spear_set_gemm_slices(int32_t k_slices) { g_ov_gs = k_slices > 0 ? k_slices : 0; }

void spear_set_gemv_stages(int32_t stages) { g_ov_nst = stages > 0 ? stages : 0; }

void spear_set_gemm_tile(int32_t tokens) { g_ov_gt = tokens == 128 || tokens == 256 ? tokens : 0; }
void spear_set_gemm_roles(int32_t roles) { g_ov_gr = roles >= 1 && roles <= 3 ? roles : 0; }

const char* spear_status_string(spear_status_t s) {
  switch (s) {
    case SPEAR_OK: return "ok";
    case SPEAR_E_NULL: return "a required pointer is NULL";
    case SPEAR_E_SHAPE: return "shape outside the supported set";
    case SPEAR_E_DTYPE: return "unknown activation dtype";
    case SPEAR_E_ALIGN: return "pointer not 16-byte aligned";
    case SPEAR_E_WORKSPACE: return "workspace missing or too small";
    case SPEAR_E_UNSUPPORTED: return "gate kind or path not supported";
    case SPEAR_E_HIP: return "HIP launch failed";
    case SPEAR_E_ALIAS: return "output overlaps an input";
    default: return "unknown status";
  }
}

const char* spear_version(void) { return "0.2.0"; }

}  // extern "C"
