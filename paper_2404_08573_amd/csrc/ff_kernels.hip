// gfx950 (CDNA4) kernels of the Forward-Forward training step and label scoring.
//
// Method: Aktemur et al., "Going Forward-Forward in Distributed Deep Learning"
// (arXiv 2404.08573), Sec. 3 (goodness, Eq. 1; prediction), Sec. 5.1 (layers, Adam).
//
// Kernels
//   k_embed_norm   label embedding (Sec. 3 "Negative Data") + row L2 normalisation;
//                  one wave per row, float4 loads, HBM-bound.
//   k_fwd          Z = X W^T on MFMA (v_mfma_f32_32x32x2f32 for fp32 operands,
//                  v_mfma_f32_32x32x16_bf16 for bf16), operands loaded straight into
//                  LDS (buffer_load ... lds); the epilogue fuses bias, ReLU, the
//                  H store and the per-row goodness partial sum over the tile's
//                  columns (Eq. 1) through a lane butterfly and LDS.
//   k_loss_rows    goodness partials -> g, the per-row gradient coefficient
//                  c_r = 2 dL/dg_r and per-workgroup sums of the Eq. 1 loss terms.
//   k_dw_adam_f32  dW = (c.H)^T X_hat on fp32 MFMA (contraction over the batch rows),
//                  the row scale c applied while staging H, db summed from the same
//                  staged rows, and the Adam update of W and b fused in the epilogue
//                  (no split over rows, so every dW tile is final in one workgroup);
//                  its first thread also finishes the loss scalar in a fixed order.
//   k_dw_adam_bf16 the same on v_mfma_f32_32x32x16_bf16: tiles staged in their
//                  natural layout, MFMA fragments through LDS transpose reads.
//   k_goodness, k_argmax, k_bf16_shadow: small row/elementwise kernels.
//
// Every reduction runs in a fixed order, so results are bitwise reproducible
// run to run and independent of stream interleaving.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <type_traits>

#include "ff_internal.h"

namespace ffk {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kBlock = 256;  // 4 waves of 64 lanes

__device__ __forceinline__ float4 ld4(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ uint4 ld16(const void *p) { return *reinterpret_cast<const uint4 *>(p); }
__device__ __forceinline__ void st16(void *p, uint4 v) { *reinterpret_cast<uint4 *>(p) = v; }
__device__ __forceinline__ float4 as_f4(uint4 u) {
  return make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z),
                     __uint_as_float(u.w));
}
__device__ __forceinline__ bf16x8 as_bf8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ float comp(const float4 &v, int q) {
  return q == 0 ? v.x : (q == 1 ? v.y : (q == 2 ? v.z : v.w));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> packed bf16 (a in the low half), round to nearest even; gfx950
// does this in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint16_t bf16_of(float a) {
  return __builtin_bit_cast(uint16_t, (__bf16)a);
}
__device__ __forceinline__ float bf16_round_f(float a) { return (float)(__bf16)a; }
__device__ __forceinline__ float bf16_bits_to_f(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ float softplus_f(float x) {
  return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x)));
}
__device__ __forceinline__ float sigmoid_f(float x) {
  const float e = expf(-fabsf(x));
  return x >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
}

// One Adam update: m, v moments; p -= lr m_hat / (sqrt(v_hat) + eps).  The
// square root and the reciprocal are the hardware's (about 1 ulp each, far
// below what the update's fp32 inputs carry): the IEEE-exact sequences cost
// several times the instructions, which matters in the one-wave-per-SIMD
// epilogues that run this for every weight.
__device__ __forceinline__ void adam_update(float &p, float &m, float &v, float g,
                                            const AdamArgs &a) {
  m = a.beta1 * m + (1.f - a.beta1) * g;
  v = a.beta2 * v + (1.f - a.beta2) * g * g;
  p = p - a.lr_bc1 * m * __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(v * a.inv_bc2) + a.eps);
}

// ---------------------------------------------------------------------------
// Row source mapping (label embedding) + L2 normalisation
// ---------------------------------------------------------------------------
constexpr int kNeutralLab = -2;

__device__ __forceinline__ void map_row(const RowMap &m, int r, int &src, int &lab) {
  if (m.mode == PAIRS) {
    if (r < m.n_pos) {
      src = m.base_off + r;
      lab = m.lab_a[src];
    } else {
      src = m.base_off + r - m.n_pos;
      lab = m.lab_b[src];
    }
  } else if (m.mode == EXPAND) {
    src = m.base_off + r / m.n_classes;
    lab = r % m.n_classes;
  } else if (m.mode == MASKED) {
    src = m.base_off + r;
    lab = m.n_classes;  // matches no label feature: all of them become 0
  } else if (m.mode == NEUTRAL) {
    src = m.base_off + r;
    lab = kNeutralLab;
  } else {
    src = r;
    lab = -1;
  }
}

// Features [col, col+4) of a row under label `lab`: the first C features are
// replaced by one-hot(lab) (all zero when lab >= C), or all set to the neutral
// 0.1 (lab == kNeutralLab); other negative labels leave the row as is.
__device__ __forceinline__ float4 embed4(float4 v, int col, int lab, int C) {
  if (lab == kNeutralLab && col < C) {
    v.x = col + 0 < C ? 0.1f : v.x;
    v.y = col + 1 < C ? 0.1f : v.y;
    v.z = col + 2 < C ? 0.1f : v.z;
    v.w = col + 3 < C ? 0.1f : v.w;
  } else if (lab >= 0 && col < C) {
    v.x = col + 0 < C ? (col + 0 == lab ? 1.f : 0.f) : v.x;
    v.y = col + 1 < C ? (col + 1 == lab ? 1.f : 0.f) : v.y;
    v.z = col + 2 < C ? (col + 2 == lab ? 1.f : 0.f) : v.z;
    v.w = col + 3 < C ? (col + 3 == lab ? 1.f : 0.f) : v.w;
  }
  return v;
}

template <bool BF16OUT>
__global__ __launch_bounds__(kBlock) void k_embed_norm(RowMap m, int rows, int d, float eps,
                                                       int normalise, void *out,
                                                       float *scale_out) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (r >= rows) return;  // uniform per wave
  int src, lab;
  map_row(m, r, src, lab);
  const float *xr = m.base + (size_t)src * d;
  const int d4 = d >> 2;
  float scale = 1.f;
  if (normalise) {
    float ss = 0.f;
    for (int i = lane; i < d4; i += 64) {
      const float4 v = embed4(ld4(xr + 4 * i), 4 * i, lab, m.n_classes);
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    ss = wave_sum(ss);
    if (m.mode == MASKED) ss += 1.f;  // the one-hot label feature every embedding carries
    scale = 1.f / (sqrtf(ss) + eps);
  }
  if (scale_out && lane == 0) scale_out[r] = BF16OUT ? bf16_round_f(scale) : scale;
  for (int i = lane; i < d4; i += 64) {
    float4 v = embed4(ld4(xr + 4 * i), 4 * i, lab, m.n_classes);
    v.x *= scale;
    v.y *= scale;
    v.z *= scale;
    v.w *= scale;
    if (BF16OUT) {
      uint2 p;
      p.x = pack_bf16(v.x, v.y);
      p.y = pack_bf16(v.z, v.w);
      reinterpret_cast<uint2 *>(out)[(size_t)r * d4 + i] = p;
    } else {
      st4(reinterpret_cast<float *>(out) + (size_t)r * d + 4 * i, v);
    }
  }
}

// The same for rows of at most 256 * NV features, held in registers: each
// lane issues its NV float4 loads before using any, so a wave keeps NV KB in
// flight, and the row is read once (the general kernel above reads it twice
// and waits on each load in turn).
template <int NV, bool BF16OUT>
__global__ __launch_bounds__(kBlock) void k_embed_norm_reg(RowMap m, int rows, int d, float eps,
                                                           int normalise, void *out,
                                                           float *scale_out) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  if (r >= rows) return;  // uniform per wave
  int src, lab;
  map_row(m, r, src, lab);
  const float *xr = m.base + (size_t)src * d;
  const int d4 = d >> 2;
  float4 v[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = lane + 64 * j;
    v[j] = i < d4 ? ld4(xr + 4 * i) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    v[j] = embed4(v[j], 4 * (lane + 64 * j), lab, m.n_classes);
    ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
  }
  float scale = 1.f;
  if (normalise) {
    ss = wave_sum(ss);
    if (m.mode == MASKED) ss += 1.f;  // the one-hot label feature every embedding carries
    scale = 1.f / (sqrtf(ss) + eps);
  }
  if (scale_out && lane == 0) scale_out[r] = BF16OUT ? bf16_round_f(scale) : scale;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = lane + 64 * j;
    if (i >= d4) break;
    const float4 t = make_float4(v[j].x * scale, v[j].y * scale, v[j].z * scale, v[j].w * scale);
    if (BF16OUT) {
      uint2 p;
      p.x = pack_bf16(t.x, t.y);
      p.y = pack_bf16(t.z, t.w);
      reinterpret_cast<uint2 *>(out)[(size_t)r * d4 + i] = p;
    } else {
      st4(reinterpret_cast<float *>(out) + (size_t)r * d + 4 * i, t);
    }
  }
}

// ---------------------------------------------------------------------------
// Reduce-scatter of NV per-lane values over the 32 lanes of each half-wave
// (butterfly: at each step a lane keeps one half of its array and adds the
// partner's copy of that half).  On return, for NV >= 32, lane l holds in
// v[j], j < NV/32, the full sum of entry j + (NV/32)*(l & 31); for NV == 16
// it holds in v[0] the sum of entry (l & 31) >> 1 (lanes l and l^1 agree).
// ---------------------------------------------------------------------------
template <int NV>
__device__ __forceinline__ void rowsum_scatter(float (&v)[NV], int lane) {
  static_assert(NV == 16 || NV == 32 || NV == 64, "16, 32 or 64 values");
  constexpr int kSteps = NV == 16 ? 4 : 5;
#pragma unroll
  for (int st = 0, o = 16, half = NV / 2; st < kSteps; ++st, o >>= 1, half >>= 1) {
    const bool hi = (lane & o) != 0;
#pragma unroll
    for (int q = 0; q < half; ++q) {
      float lo = v[q], up = v[q + half];
      // Both halves as register values before the selects: left as selects
      // between array elements, they were compiled as indexed accesses into
      // the whole array (a 500-instruction select network per kernel, or the
      // array moved out of registers).
      asm volatile("" : "+v"(lo), "+v"(up));
      const float send = hi ? lo : up;
      const float keep = hi ? up : lo;
      v[q] = keep + __shfl_xor(send, o);
    }
  }
  if (NV == 16) v[0] += __shfl_xor(v[0], 1);
}

// XCD-aware tile order.  Workgroups are dealt round-robin to the 8 XCDs, each
// with its own L2, so consecutive workgroup ids land on different L2s.  Each
// XCD is given a contiguous range of tiles instead, walked in groups of G row
// panels (all column panels of a group before the next group), so the
// workgroups sharing an L2 at a given time also share operand panels.  A
// bijection of tile indices: results do not depend on it.
__device__ __forceinline__ void tile_of(int bid, int mt, int nt, int &tm, int &tn) {
  constexpr int kXcd = 8, G = 4;
  const int T = mt * nt;
  const int q = T / kXcd, r = T % kXcd;
  const int x = bid % kXcd, j = bid / kXcd;
  const int t = x * q + min(x, r) + j;
  const int gsz = G * nt;
  const int g = t / gsz, o = t % gsz;
  const int rows = min(G, mt - g * G);
  tm = g * G + o % rows;
  tn = o / rows;
}

// Row (within a 32x32 block) of accumulator register r held by a lane of
// half-wave kg: the v_mfma_f32_32x32x2f32 output layout puts row
// 8*(r/4) + 4*kg + r%4 in register r (column = lane % 32).
__device__ __forceinline__ int acc_row(int r, int kg) { return 8 * (r >> 2) + 4 * kg + (r & 3); }

// V consecutive floats from LDS (V = 1, 2 or 4) as an array.
template <int V>
__device__ __forceinline__ void lds_vec(const float *p, float (&out)[V]) {
  if constexpr (V == 4) {
    const float4 t = ld4(p);
    out[0] = t.x;
    out[1] = t.y;
    out[2] = t.z;
    out[3] = t.w;
  } else if constexpr (V == 2) {
    const float2 t = *reinterpret_cast<const float2 *>(p);
    out[0] = t.x;
    out[1] = t.y;
  } else {
    out[0] = p[0];
  }
}

// Workgroup barrier that the compiler may not move memory accesses across.
// The s_barrier builtin alone is no memory fence, so LDS reads of a tile could
// be scheduled across it, and __syncthreads' workgroup fence would also wait
// for every outstanding load into LDS (vmcnt(0)), draining the prefetch.  The
// empty asm statements with a memory clobber pin the order at the compiler
// level; the hardware order comes from the explicit s_waitcnt before it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt operand: at most n vector-memory operations outstanding, no limit
// on the other counters (gfx9 encoding: vmcnt in bits 3:0 and 15:14).
constexpr int vmcnt_wait(int n) { return 0x0f70 | (n & 15) | ((n >> 4) << 14); }
// s_waitcnt operands: nothing outstanding; no LDS (or scalar memory) operation
// outstanding, any number of vector-memory ones.
constexpr int kWaitAll = 0x0070;
constexpr int kWaitLds = 0xc07f;

// Software pipeline over nk k-tiles with double-buffered LDS and PF register
// stages: the loads of tile t+PF are issued before the MFMAs of tile t, and
// tile t+1 is written from its register stage to the other LDS buffer after
// them.  Load results are consumed only there, so each load has PF tiles of
// MFMA work to land.  The steady-state body is straight-line code (loads and
// LDS writes unconditional: loads past the last tile read clamped valid
// addresses and are masked to zero, and their LDS buffer is never read), so
// the compiler's wait counters track each stage separately instead of
// draining every load at a control-flow join.  The loop is unrolled by
// lcm(PF, 2) so that register stages and LDS buffers are fixed; each LDS
// buffer is rewritten only after the barrier that ends the computation
// reading it, and each register stage only after it has been written to LDS.
//
// The barrier after each LDS write waits for the thread's own LDS writes
// only (lgkmcnt(0)): __syncthreads' workgroup fence would also wait for every
// outstanding global load, the register stages of the next PF - 1 tiles, and
// so cut the prefetch to the tile issued in the same iteration.
template <int PF, class Load, class Store, class Compute, class Stage>
__device__ __forceinline__ void kloop(int nk, Load &gload, Store &sstore, Compute &compute,
                                      Stage (&st)[PF]) {
  constexpr int U = PF % 2 == 0 ? PF : 2 * PF;
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(kWaitLds);
    lds_barrier();
  };
#pragma unroll
  for (int j = 0; j < PF; ++j) gload(st[j], j);
  sstore(st[0], 0);
  barrier();
  int kt = 0;
  for (; kt + U <= nk; kt += U) {
#pragma unroll
    for (int j = 0; j < U; ++j) {
      gload(st[j % PF], kt + j + PF);
      compute(j % 2);
      sstore(st[(j + 1) % PF], (j + 1) % 2);
      barrier();
    }
  }
#pragma unroll
  for (int j = 0; j < U; ++j) {
    if (kt + j < nk) {
      gload(st[j % PF], kt + j + PF);
      compute(j % 2);
      sstore(st[(j + 1) % PF], (j + 1) % 2);
      barrier();
    }
  }
  __builtin_amdgcn_s_waitcnt(kWaitAll);  // the loads past the last tile, before the LDS is reused
}

// ---------------------------------------------------------------------------
// Forward: H = relu(X W^T + b), gpart[tn][row] = sum over the tile's columns of H^2.
// X [M][K], W [N][K] (both K-contiguous), fp32 or bf16 operands, fp32
// accumulation.  Tile BM x BN, WM x WN waves, each (BM/WM) x (BN/WN) as 32x32
// MFMA blocks: v_mfma_f32_32x32x2f32 (one fp32 per lane per instruction) or
// v_mfma_f32_32x32x16_bf16 (eight bf16 per lane).  Within a k-tile the two
// half-waves take the two halves of its k range, so every lane reads
// contiguous 16-byte runs from LDS for both operands (the k order inside the
// contraction is a permutation of the plain order, the same for X and W).
// K must be a multiple of the 16-byte vector (4 fp32 / 8 bf16).
// ---------------------------------------------------------------------------
template <bool BF16>
struct Operand;
template <>
struct Operand<false> {
  using T = float;
  static constexpr int kVec = 4;  // elements per 16 bytes
};
template <>
struct Operand<true> {
  using T = uint16_t;  // bf16 bits
  static constexpr int kVec = 8;
};

// A k-tile of the NT main loop is 128 bytes of every operand row.
template <bool BF16>
constexpr int nt_bk() {
  return 128 / (int)sizeof(typename Operand<BF16>::T);
}
// LDS elements of the NT main loop's NBUF-stage tiles.
template <bool BF16, int BM, int BN, int NBUF>
constexpr int nt_lds_elems() {
  return NBUF * (BM + BN) * nt_bk<BF16>();
}

typedef __attribute__((address_space(3))) void lds_void;

// Raw buffer descriptor over `bytes` bytes from `base`: loads at offsets at or
// past `bytes` return zeros instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                           0x00020000);
}
constexpr uint32_t kOutOfRange = 0x80000000u;  // a buffer offset past every tile's range

// LDS position of 16-byte chunk c of tile row r in its unpadded 128-byte row.
// The MFMA fragment reads take one chunk on 16 consecutive rows per group of
// 16 lanes; this XOR puts them on 16 distinct 16-byte positions modulo 256
// bytes (two rows share a 256-byte line of the 64 banks, so rows r and r + 8
// are told apart by bit 3 of r) and on 8 distinct positions within every 8
// rows.  An involution for each r.
__device__ __forceinline__ int nt_swz(int r, int c) { return c ^ (r & 7) ^ ((r >> 3) & 1); }


// Main loop of C[m][n] = sum_k X[m][k] W[n][k] for the tile at (m0, n0), both
// operands K-contiguous, into the wave's accumulators.
//
// Operands move from global memory straight into LDS (buffer_load ... lds,
// 16 bytes per lane): one wave instruction fills 8 unpadded 128-byte tile
// rows, lane l writing LDS position l % 8 of row l / 8 and fetching the chunk
// that nt_swz maps to that position.  The buffer descriptors span the tile's
// valid rows, so rows past M or N and chunks past K (the k tail, given an
// out-of-range offset) arrive as zeros.  NBUF LDS stages: the loads of tile
// t + NBUF - 1 are issued right after the barrier that opens tile t (which
// ends every wave's reads of tile t - 1, whose buffer they refill), and tile
// t's own loads are waited for by counter before that barrier, so NBUF - 2
// tiles of loads stay in flight across the MFMAs.  Loads past the last tile
// are issued all the same (they read zeros), keeping the counter arithmetic
// exact.  On return every load has landed and every wave has passed a
// barrier, so the LDS may be reused.  The descriptors' 32-bit range needs
// min(BM, M - m0) * K and min(BN, N - n0) * K under 2^31 bytes.
template <bool BF16, int BM, int BN, int WM, int WN, int NBUF>
__device__ __forceinline__ void nt_mainloop(const typename Operand<BF16>::T *__restrict__ X,
                                            const typename Operand<BF16>::T *__restrict__ W,
                                            int M, int N, int K, int m0, int n0,
                                            typename Operand<BF16>::T *sm,
                                            floatx16 (&acc)[BM / WM / 32][BN / WN / 32]) {
  using T = typename Operand<BF16>::T;
  constexpr int VE = Operand<BF16>::kVec;
  constexpr int ES = sizeof(T);
  constexpr int BK = nt_bk<BF16>();
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  constexpr int IA = BM / 8 / NW, IB = BN / 8 / NW;  // 8-row wave loads per k-tile
  constexpr int STAGE = (BM + BN) * BK;               // elements per LDS stage
  static_assert(MB * 32 == TM && NB * 32 == TN, "wave tile is whole 32x32 blocks");
  static_assert(IA * 8 * NW == BM && IB * 8 * NW == BN, "tile rows split into 8-row wave loads");
  static_assert(NBUF >= 2 && (NBUF - 2) * (IA + IB) < 64, "stages");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;

  const __amdgpu_buffer_rsrc_t ra =
      buffer_rsrc(X + (size_t)m0 * K, (uint32_t)(min(BM, M - m0) * K * ES));
  const __amdgpu_buffer_rsrc_t rb =
      buffer_rsrc(W + (size_t)n0 * K, (uint32_t)(min(BN, N - n0) * K * ES));
  const int lpos = lane & 7;
  int kca[IA], kcb[IB];   // element offset of the lane's chunk within a k-tile
  uint32_t oa[IA], ob[IB];  // byte offset of that chunk in k-tile 0
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r = (wave * IA + i) * 8 + (lane >> 3);
    kca[i] = nt_swz(r, lpos) * VE;
    oa[i] = (uint32_t)((r * K + kca[i]) * ES);
  }
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r = (wave * IB + i) * 8 + (lane >> 3);
    kcb[i] = nt_swz(r, lpos) * VE;
    ob[i] = (uint32_t)((r * K + kcb[i]) * ES);
  }
  auto issue = [&](int kt, int buf) {
    T *As = sm + buf * STAGE;
    T *Bs = As + BM * BK;
    const int kb = kt * BK;
#pragma unroll
    for (int i = 0; i < IA; ++i) {
      // The offset goes through a typed local: with a template-dependent
      // expression as the argument, hipcc's host pass drops the kernel's
      // launch stub without a diagnostic (the library then fails to load).
      const uint32_t o = kb + kca[i] < K ? oa[i] + kb * ES : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(As + (wave * IA + i) * 8 * BK), 16,
                                               o, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < IB; ++i) {
      const uint32_t o = kb + kcb[i] < K ? ob[i] + kb * ES : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void *)(Bs + (wave * IB + i) * 8 * BK), 16,
                                               o, 0, 0, 0);
    }
  };

#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  auto compute = [&](int buf) {
    const T *As = sm + buf * STAGE;
    const T *Bs = As + BM * BK;
#pragma unroll
    for (int sv = 0; sv < BK / 2; sv += VE) {
      const int c = (kg * (BK / 2) + sv) / VE;
      uint4 a[MB], b[NB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int r = wm * TM + mb * 32 + li;
        a[mb] = ld16(As + r * BK + nt_swz(r, c) * VE);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int r = wn * TN + nb * 32 + li;
        b[nb] = ld16(Bs + r * BK + nt_swz(r, c) * VE);
      }
      if constexpr (BF16) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf8(a[mb]), as_bf8(b[nb]),
                                                                  acc[mb][nb], 0, 0, 0);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                  comp(as_f4(a[mb]), q), comp(as_f4(b[nb]), q), acc[mb][nb], 0, 0, 0);
      }
    }
  };

  const int nk = (K + BK - 1) / BK;
#pragma unroll
  for (int j = 0; j < NBUF - 1; ++j) issue(j, j);
  for (int kt = 0; kt < nk; ++kt) {
    __builtin_amdgcn_s_waitcnt(vmcnt_wait((NBUF - 2) * (IA + IB)));
    lds_barrier();
    issue(kt + NBUF - 1, (kt + NBUF - 1) % NBUF);
    compute(kt % NBUF);
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
  lds_barrier();
}

template <bool BF16, int BM, int BN, int WM, int WN, int NBUF, bool STORE_H>
__global__ __launch_bounds__(WM *WN * 64) void k_fwd(const typename Operand<BF16>::T *__restrict__ X,
                                                     const typename Operand<BF16>::T *__restrict__ W,
                                                     const float *__restrict__ bias,
                                                     const float *__restrict__ rowscale, int M,
                                                     int N, int K, float *__restrict__ H,
                                                     float *__restrict__ gpart) {
  using T = typename Operand<BF16>::T;
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  __shared__ __attribute__((aligned(16))) T sm[nt_lds_elems<BF16, BM, BN, NBUF>()];
  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;

  floatx16 acc[MB][NB];
  nt_mainloop<BF16, BM, BN, WM, WN, NBUF>(X, W, M, N, K, m0, n0, sm, acc);

  // Epilogue: row scale (the input rows' normalisation, when the operand rows
  // are raw), bias, ReLU, H store, goodness partials.
  float hsq[MB * 16], rs[MB * 16];
#pragma unroll
  for (int q = 0; q < MB * 16; ++q) {
    hsq[q] = 0.f;
    rs[q] = rowscale ? rowscale[min(m0 + wm * TM + (q >> 4) * 32 + acc_row(q & 15, kg), M - 1)]
                     : 1.f;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = n0 + wn * TN + nb * 32 + li;
    const bool cok = col < N;
    const float bv = cok ? bias[col] : 0.f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float h = cok ? fmaxf(fmaf(acc[mb][nb][r], rs[mb * 16 + r], bv), 0.f) : 0.f;
        if (STORE_H) {
          const int row = m0 + wm * TM + mb * 32 + acc_row(r, kg);
          if (row < M && cok) H[(size_t)row * N + col] = h;
        }
        hsq[mb * 16 + r] += h * h;
      }
  }
  rowsum_scatter(hsq, lane);
  float *gs = reinterpret_cast<float *>(sm);  // [WN][BM]; the main-loop buffers are free now
  if constexpr (MB == 1) {
    const int q = (lane & 31) >> 1;
    if ((lane & 1) == 0) gs[wn * BM + wm * TM + acc_row(q, kg)] = hsq[0];
  } else {
#pragma unroll
    for (int j = 0; j < MB / 2; ++j) {
      const int q = j + (MB / 2) * (lane & 31);
      gs[wn * BM + wm * TM + (q >> 4) * 32 + acc_row(q & 15, kg)] = hsq[j];
    }
  }
  __syncthreads();
  for (int t = tid; t < BM; t += NT) {
    const int row = m0 + t;
    if (row < M) {
      float g = 0.f;
#pragma unroll
      for (int w = 0; w < WN; ++w) g += gs[w * BM + t];
      gpart[(size_t)tn * M + row] = g;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 forward on four waves of 128 x (BN/2) each (one wave per SIMD).
// The 8-wave tiles above give each wave a 32x64 or 64x96 share, whose MFMA
// fragments cost more LDS read bytes per flop than the CU's LDS delivers at
// the bf16 MFMA rate.  A 128x96 wave tile needs 7 fragment reads per 12
// MFMAs.  Its 192 accumulators live in AGPRs, so one wave fills a SIMD and
// must hide its own latencies:
//   * fragments are double-buffered in registers: the reads of k-step s+1
//     are issued one beside each MFMA of k-step s (sched_group_barrier);
//   * one barrier per 64-deep k-tile, placed after the first MFMA of its last
//     k-step, so the MFMA pipe is busy while the waves meet;
//   * after that barrier, the loads of k-tile t+2 and the first fragments of
//     k-tile t+1 are issued one slot per MFMA of the rest of that k-step.
// Same operand layout, k permutation, swizzle and zero-filled tails as
// nt_mainloop with two LDS stages; same epilogue results as k_fwd.
// ---------------------------------------------------------------------------

// s_waitcnt operand: at most n vector-memory operations and no LDS operation
// outstanding.
constexpr int vmcnt_lgkm0(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

template <int BM, int BN, int NBUF = 2>
__device__ __forceinline__ void nt_mainloop4(const uint16_t *__restrict__ X,
                                             const uint16_t *__restrict__ W, int M, int N, int K,
                                             int m0, int n0, uint16_t *sm,
                                             floatx16 (&acc)[BM / 64][BN / 64]) {
  constexpr int VE = 8, ES = 2, BK = 64, NW = 4, WN = 2;
  constexpr int TM = BM / 2, TN = BN / 2, MB = TM / 32, NB = TN / 32;
  constexpr int IA = BM / 8 / NW, IB = BN / 8 / NW;  // 8-row wave loads per k-tile
  constexpr int STAGE = (BM + BN) * BK;
  constexpr int KS = BK / 2 / VE;  // 16-deep k-steps per k-tile
  // the last k-step of a k-tile has NM MFMAs after its barrier and ND
  // fragment reads of the next k-tile: NS slots carry them with the loads
  constexpr int NM = MB * NB - 1, ND = MB + NB, NV = IA + IB, NS = NM > ND ? NM : ND;
  static_assert(MB * 32 == TM && NB * 32 == TN && IA * 8 * NW == BM && IB * 8 * NW == BN,
                "tile shape");
  static_assert(ND <= MB * NB && KS % 2 == 0, "a fragment read per MFMA");
  static_assert(NBUF >= 2 && (NBUF - 1) * (IA + IB) < 64, "stages");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;
  const __amdgpu_buffer_rsrc_t ra =
      buffer_rsrc(X + (size_t)m0 * K, (uint32_t)(min(BM, M - m0) * K * ES));
  const __amdgpu_buffer_rsrc_t rb =
      buffer_rsrc(W + (size_t)n0 * K, (uint32_t)(min(BN, N - n0) * K * ES));
  const int lpos = lane & 7;
  int kca[IA], kcb[IB];
  uint32_t oa[IA], ob[IB];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r = (wave * IA + i) * 8 + (lane >> 3);
    kca[i] = nt_swz(r, lpos) * VE;
    oa[i] = (uint32_t)((r * K + kca[i]) * ES);
  }
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r = (wave * IB + i) * 8 + (lane >> 3);
    kcb[i] = nt_swz(r, lpos) * VE;
    ob[i] = (uint32_t)((r * K + kcb[i]) * ES);
  }
  // Load j of k-tile kt into stage buf: 8 rows of the X tile for j < IA, else
  // 8 rows of the W tile.
  auto issue1 = [&](int kt, int buf, int j) {
    uint16_t *As = sm + buf * STAGE;
    const int kb = kt * BK;
    if (j < IA) {
      const uint32_t o = kb + kca[j] < K ? oa[j] + kb * ES : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(As + (wave * IA + j) * 8 * BK), 16,
                                               o, 0, 0, 0);
    } else {
      const int i = j - IA;
      const uint32_t o = kb + kcb[i] < K ? ob[i] + kb * ES : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rb, (lds_void *)(As + BM * BK + (wave * IB + i) * 8 * BK), 16, o, 0, 0, 0);
    }
  };
  // LDS offsets (elements) of the lane's fragment rows in stage 0.
  int pa[MB], pb[NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) pa[mb] = (wm * TM + mb * 32 + li) * BK;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) pb[nb] = BM * BK + (wn * TN + nb * 32 + li) * BK;
  // Fragment i of k-step ks from stage buf: X block i for i < MB, else W block i - MB.
  auto rd1 = [&](int buf, int ks, int i, uint4 (&a)[MB], uint4 (&b)[NB]) {
    const uint16_t *S = sm + buf * STAGE;
    const int c = kg * KS + ks;
    if (i < MB)
      a[i] = ld16(S + pa[i] + nt_swz(i * 32 + li, c) * VE);
    else
      b[i - MB] = ld16(S + pb[i - MB] + nt_swz((i - MB) * 32 + li, c) * VE);
  };
  auto mm = [&](int mb, int nb, const uint4 &a, const uint4 &b) {
    acc[mb][nb] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf8(a), as_bf8(b), acc[mb][nb], 0, 0, 0);
  };
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  uint4 fa[2][MB], fb[2][NB];
  const int nk = (K + BK - 1) / BK;
  // NBUF LDS stages: k-tiles 0..NBUF-1 are issued up front; k-tile kt + NBUF
  // goes into k-tile kt's stage after the barrier that ends kt's reads, so
  // NBUF - 1 k-tiles stay in flight beside the MFMAs.
#pragma unroll
  for (int b = 0; b < NBUF; ++b)
#pragma unroll
    for (int j = 0; j < NV; ++j) issue1(b, b, j);
  __builtin_amdgcn_s_waitcnt(vmcnt_wait((NBUF - 1) * NV));
  lds_barrier();
#pragma unroll
  for (int i = 0; i < ND; ++i) rd1(0, 0, i, fa[0], fb[0]);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt % NBUF, bnext = (kt + 1) % NBUF;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1, nxt = cur ^ 1;
      if (ks + 1 < KS) {
#pragma unroll
        for (int i = 0; i < ND; ++i) rd1(buf, ks + 1, i, fa[nxt], fb[nxt]);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) mm(mb, nb, fa[cur][mb], fb[cur][nb]);
        // One fragment read beside each MFMA, the rest of the MFMAs after.
#pragma unroll
        for (int i = 0; i < ND; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        }
        __builtin_amdgcn_sched_group_barrier(0x008, MB * NB - ND, 0);
        __builtin_amdgcn_sched_barrier(0);
      } else {
        mm(0, 0, fa[cur][0], fb[cur][0]);
        __builtin_amdgcn_sched_barrier(0);
        // Every fragment of k-tile kt is in registers and k-tile kt + 1 has
        // landed (the loads of the NBUF - 2 tiles after it may still be in
        // flight): one barrier opens kt + 1 and frees kt's stage for kt + NBUF.
        __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0((NBUF - 2) * NV));
        lds_barrier();
        __builtin_amdgcn_sched_barrier(0);
        // Slots of (loads, one fragment read, one MFMA), kept in this order.
#pragma unroll
        for (int i = 0; i < NS; ++i) {
#pragma unroll
          for (int j = (i * NV) / NS; j < ((i + 1) * NV) / NS; ++j) issue1(kt + NBUF, buf, j);
          if (i < ND) rd1(bnext, 0, i, fa[nxt], fb[nxt]);
          if (i < NM) {
            const int p = i + 1;
            mm(p / NB, p % NB, fa[cur][p / NB], fb[cur][p % NB]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));
  lds_barrier();
}

template <int BM, int BN, int NBUF, bool STORE_H>
__global__ __launch_bounds__(256) void k_fwd4(const uint16_t *__restrict__ X,
                                              const uint16_t *__restrict__ W,
                                              const float *__restrict__ bias,
                                              const float *__restrict__ rowscale, int M, int N,
                                              int K, float *__restrict__ H,
                                              float *__restrict__ gpart) {
  constexpr int WN = 2, TM = BM / 2, TN = BN / 2, MB = TM / 32, NB = TN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t sm[NBUF * (BM + BN) * 64];
  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;
  floatx16 acc[MB][NB];
  nt_mainloop4<BM, BN, NBUF>(X, W, M, N, K, m0, n0, sm, acc);

  // Epilogue as in k_fwd, one 32-row block at a time, so that only 16 row
  // sums and scales are live beside the accumulators.
  float bv[NB];
  bool cok[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = n0 + wn * TN + nb * 32 + li;
    cok[nb] = col < N;
    bv[nb] = cok[nb] ? bias[col] : 0.f;
  }
  float *gs = reinterpret_cast<float *>(sm);  // [WN][BM]; the main-loop buffers are free now
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    float hsq[16], rs[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      hsq[r] = 0.f;
      rs[r] = rowscale ? rowscale[min(m0 + wm * TM + mb * 32 + acc_row(r, kg), M - 1)] : 1.f;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int col = n0 + wn * TN + nb * 32 + li;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float h = cok[nb] ? fmaxf(fmaf(acc[mb][nb][r], rs[r], bv[nb]), 0.f) : 0.f;
        if (STORE_H) {
          const int row = m0 + wm * TM + mb * 32 + acc_row(r, kg);
          if (row < M && cok[nb]) H[(size_t)row * N + col] = h;
        }
        hsq[r] += h * h;
      }
    }
    rowsum_scatter(hsq, lane);
    const int q = (lane & 31) >> 1;
    if ((lane & 1) == 0) gs[wn * BM + wm * TM + mb * 32 + acc_row(q, kg)] = hsq[0];
  }
  __syncthreads();
  for (int t = tid; t < BM; t += 256) {
    const int row = m0 + t;
    if (row < M) gpart[(size_t)tn * M + row] = gs[t] + gs[BM + t];
  }
}

// ---------------------------------------------------------------------------
// bf16 weight gradient on the four-wave main loop: dW = dZ^T (x_hat^T)^T over
// the Rp rows (both operands row-major over the rows, from k_loss_t: its loss
// workgroups write dZ^T, its transposing ones x_hat^T, or the previous layer's
// loss pass handed x_hat^T over), with the Adam update of W, its bf16 shadow and
// (column tile 0) of b fused in the epilogue; the first workgroup also finishes
// the loss.  The accumulators go through LDS half a tile at a time (the rows of
// the waves with wm = 0, then wm = 1), and each thread keeps kAdamBatch
// float4 updates' loads in flight, so the W, m, v traffic streams instead of
// waiting on one load at a time.  db sums the 64-row column partials of
// k_loss_t in a fixed order.
// ADAM = false: the epilogue stores dW (fp32, [M][N]) into G instead, and
// k_adam_dense applies the same update (and the one of b) in a launch of its
// own, which holds no LDS and so shares the CUs with other streams' products.
// ---------------------------------------------------------------------------
constexpr int kAdamBatch = 6;
// k_adam_dense keeps 3 groups in flight: at 64 VGPRs a wave of it fits beside
// a wave of the four-wave forward (448 of a SIMD's 512 registers per lane) on
// the same CU, so in pipelined epochs it runs beside other layers' forwards
// too; it streams as fast alone as with 6 (3072x3072: 45 us either way).
constexpr int kAdamDenseBatch = 3;

template <int BM, int BN, int NBUF, bool ADAM>
__global__ __launch_bounds__(256) void k_dw4(const uint16_t *__restrict__ dzT,
                                             const uint16_t *__restrict__ xT, int M, int N,
                                             int K, float *__restrict__ G,
                                             float *__restrict__ W, float *__restrict__ mW,
                                             float *__restrict__ vW, uint16_t *__restrict__ Wb,
                                             const float *__restrict__ dbp, int nrb,
                                             float *__restrict__ bvec, float *__restrict__ mbv,
                                             float *__restrict__ vbv, AdamArgs ad, LossFinish lf) {
  constexpr int WN = 2, TM = BM / 2, TN = BN / 2, MB = TM / 32, NB = TN / 32;
  constexpr int LDC = BN + 4;
  constexpr int kMain = NBUF * (BM + BN) * 64;          // bf16 elements
  constexpr int kEpi = TM * LDC * 2;                    // an fp32 half tile, in bf16 elements
  __shared__ __attribute__((aligned(16))) uint16_t sm[kMain > kEpi ? kMain : kEpi];
  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;

  if (lf.loss && blockIdx.x == 0 && tid == 0) {
    float sp = 0.f, sn = 0.f;
    for (int i = 0; i < lf.nblk; ++i) {
      sp += lf.lpart[2 * i];
      sn += lf.lpart[2 * i + 1];
    }
    lf.loss[0] = sp / (float)lf.n_pos + sn / (float)lf.n_neg;
  }

  floatx16 acc[MB][NB];
  nt_mainloop4<BM, BN, NBUF>(dzT, xT, M, N, K, m0, n0, sm, acc);

  float *Cs = reinterpret_cast<float *>(sm);  // [TM][LDC]; the main-loop buffers are free
  constexpr int Q = TM * (BN / 4);            // float4 updates per half tile
#pragma unroll 1
  for (int half = 0; half < 2; ++half) {
    if (wm == half) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            Cs[(mb * 32 + acc_row(r, kg)) * LDC + wn * TN + nb * 32 + li] = acc[mb][nb][r];
    }
    __syncthreads();
    const int mh = m0 + half * TM;
#pragma unroll 1
    for (int i0 = tid; i0 < Q; i0 += 256 * kAdamBatch) {
      float4 p[kAdamBatch], m[kAdamBatch], v[kAdamBatch];
      size_t o[kAdamBatch];
      bool ok[kAdamBatch];
#pragma unroll
      for (int u = 0; u < kAdamBatch; ++u) {
        const int idx = i0 + 256 * u;
        const int mr = idx / (BN / 4), n4 = (idx % (BN / 4)) * 4;
        ok[u] = idx < Q && mh + mr < M && n0 + n4 < N;
        o[u] = ok[u] ? (size_t)(mh + mr) * N + n0 + n4 : 0;
        if (ADAM && ok[u]) {
          p[u] = ld4(W + o[u]);
          m[u] = ld4(mW + o[u]);
          v[u] = ld4(vW + o[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < kAdamBatch; ++u) {
        if (!ok[u]) continue;
        const int idx = i0 + 256 * u;
        const int mr = idx / (BN / 4), n4 = (idx % (BN / 4)) * 4;
        const float4 g = ld4(Cs + mr * LDC + n4);
        if (!ADAM) {
          st4(G + o[u], g);
          continue;
        }
        adam_update(p[u].x, m[u].x, v[u].x, g.x, ad);
        adam_update(p[u].y, m[u].y, v[u].y, g.y, ad);
        adam_update(p[u].z, m[u].z, v[u].z, g.z, ad);
        adam_update(p[u].w, m[u].w, v[u].w, g.w, ad);
        st4(W + o[u], p[u]);
        st4(mW + o[u], m[u]);
        st4(vW + o[u], v[u]);
        if (Wb) {
          uint2 sh;
          sh.x = pack_bf16(p[u].x, p[u].y);
          sh.y = pack_bf16(p[u].z, p[u].w);
          *reinterpret_cast<uint2 *>(Wb + o[u]) = sh;
        }
      }
    }
    __syncthreads();  // the half tile's reads are done before the next one is written
  }

  if (ADAM && tn == 0) {  // db = sum of the 64-row column partials, then Adam on b
    for (int t = tid; t < BM; t += 256) {
      const int row = m0 + t;
      if (row >= M) continue;
      float sum = 0.f;  // in block order, 16 loads in flight
      int k = 0;
      for (; k + 16 <= nrb; k += 16) {
        float q[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) q[j] = dbp[(size_t)(k + j) * M + row];
#pragma unroll
        for (int j = 0; j < 16; ++j) sum += q[j];
      }
      for (; k < nrb; ++k) sum += dbp[(size_t)k * M + row];
      float p = bvec[row], m = mbv[row], v = vbv[row];
      adam_update(p, m, v, sum, ad);
      bvec[row] = p;
      mbv[row] = m;
      vbv[row] = v;
    }
  }
}

// Adam on W [M][N] (and its bf16 shadow Wb) from the weight gradient G, and
// on b from the 64-row column partials dbp [nrb][M] (summed in block order):
// the update k_dw4 fuses, as a launch of its own.  The first workgroups take
// float4 groups of W, kAdamBatch per thread with their loads in flight; the
// last ceil(M / 256) take one bias row per thread.  N is a multiple of 4.
__global__ __launch_bounds__(kBlock) void k_adam_dense(const float *__restrict__ G, int M, int N,
                                                       int nmain, float *__restrict__ W,
                                                       float *__restrict__ mW,
                                                       float *__restrict__ vW,
                                                       uint16_t *__restrict__ Wb,
                                                       const float *__restrict__ dbp, int nrb,
                                                       float *__restrict__ bvec,
                                                       float *__restrict__ mbv,
                                                       float *__restrict__ vbv, AdamArgs ad) {
  const int tid = threadIdx.x;
  if ((int)blockIdx.x >= nmain) {
    const int row = (blockIdx.x - nmain) * kBlock + tid;
    if (row >= M) return;
    float sum = 0.f;  // in block order, 16 loads in flight
    int k = 0;
    for (; k + 16 <= nrb; k += 16) {
      float q[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) q[j] = dbp[(size_t)(k + j) * M + row];
#pragma unroll
      for (int j = 0; j < 16; ++j) sum += q[j];
    }
    for (; k < nrb; ++k) sum += dbp[(size_t)k * M + row];
    float p = bvec[row], m = mbv[row], v = vbv[row];
    adam_update(p, m, v, sum, ad);
    bvec[row] = p;
    mbv[row] = m;
    vbv[row] = v;
    return;
  }
  const size_t n4 = (size_t)M * N / 4;
  const size_t base = (size_t)blockIdx.x * kBlock * kAdamDenseBatch + tid;
  float4 p[kAdamDenseBatch], m[kAdamDenseBatch], v[kAdamDenseBatch], g[kAdamDenseBatch];
#pragma unroll
  for (int u = 0; u < kAdamDenseBatch; ++u) {
    const size_t i = base + (size_t)u * kBlock;
    if (i < n4) {
      g[u] = ld4(G + 4 * i);
      p[u] = ld4(W + 4 * i);
      m[u] = ld4(mW + 4 * i);
      v[u] = ld4(vW + 4 * i);
    }
  }
#pragma unroll
  for (int u = 0; u < kAdamDenseBatch; ++u) {
    const size_t i = base + (size_t)u * kBlock;
    if (i >= n4) continue;
    adam_update(p[u].x, m[u].x, v[u].x, g[u].x, ad);
    adam_update(p[u].y, m[u].y, v[u].y, g[u].y, ad);
    adam_update(p[u].z, m[u].z, v[u].z, g[u].z, ad);
    adam_update(p[u].w, m[u].w, v[u].w, g[u].w, ad);
    st4(W + 4 * i, p[u]);
    st4(mW + 4 * i, m[u]);
    st4(vW + 4 * i, v[u]);
    if (Wb) {
      uint2 sh;
      sh.x = pack_bf16(p[u].x, p[u].y);
      sh.y = pack_bf16(p[u].z, p[u].w);
      *reinterpret_cast<uint2 *>(Wb + 4 * i) = sh;
    }
  }
}

// ---------------------------------------------------------------------------
// Shared-base layer-0 forward.// ---------------------------------------------------------------------------
// Shared-base layer-0 forward.  Every label embedding of an input row has the
// same norm (one label feature is 1), so with x_hat = s * (masked row + e_label)
// the product splits into P = X_masked_hat W^T, computed once per base row on
// the main loop above, plus s * W[:, label] per label.  The epilogue expands
// each base row into its E labelled output rows: bias, ReLU, H store and the
// goodness partials of each.  The tile's label columns of W are staged in LDS
// (converted from bf16 bits in bf16 mode, where s is already bf16-rounded, so
// s * W_label is exact in fp32).
// ---------------------------------------------------------------------------
template <bool BF16, int BM, int BN, int WM, int WN, int NBUF, bool STORE_H>
__global__ __launch_bounds__(WM *WN * 64) void k_fwd_expand(
    const typename Operand<BF16>::T *__restrict__ X, const typename Operand<BF16>::T *__restrict__ W,
    const float *__restrict__ bias, LabelExpand ex, int M, int N, int K, float *__restrict__ H,
    float *__restrict__ gpart) {
  using T = typename Operand<BF16>::T;
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  constexpr int kMain = nt_lds_elems<BF16, BM, BN, NBUF>() * (int)sizeof(T) / 4;  // in floats
  constexpr int kEpi = kMaxExpand * (WN * BM + BN);
  __shared__ __attribute__((aligned(16))) float smf[kMain > kEpi ? kMain : kEpi];
  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;
  const int C = ex.n_classes;

  floatx16 acc[MB][NB];
  nt_mainloop<BF16, BM, BN, WM, WN, NBUF>(X, W, M, N, K, m0, n0, reinterpret_cast<T *>(smf), acc);

  // LDS after the main loop: gs [C][WN][BM] goodness partials, wl [BN][kMaxExpand]
  // the tile's label columns of W.
  float *gs = smf;
  float *wl = smf + kMaxExpand * WN * BM;
  for (int i = tid; i < BN * C; i += NT) {
    const int j = i / C, c = i % C;
    const int col = min(n0 + j, N - 1);
    if constexpr (BF16)
      wl[j * kMaxExpand + c] = bf16_bits_to_f(W[(size_t)col * K + c]);
    else
      wl[j * kMaxExpand + c] = W[(size_t)col * K + c];
  }
  __syncthreads();

  const int rbase = m0 + wm * TM;
  float sr[MB * 16];
#pragma unroll
  for (int q = 0; q < MB * 16; ++q)
    sr[q] = ex.scale[min(rbase + (q >> 4) * 32 + acc_row(q & 15, kg), M - 1)];

  for (int c = 0; c < C; ++c) {
    float hsq[MB * 16];
#pragma unroll
    for (int q = 0; q < MB * 16; ++q) hsq[q] = 0.f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int cl = wn * TN + nb * 32 + li;
      const int col = n0 + cl;
      const bool cok = col < N;
      const float bv = cok ? bias[col] : 0.f;
      const float wc = wl[cl * kMaxExpand + c];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int q = mb * 16 + r;
          const int row = rbase + mb * 32 + acc_row(r, kg);
          const float h = cok ? fmaxf(acc[mb][nb][r] + fmaf(sr[q], wc, bv), 0.f) : 0.f;
          if (STORE_H && cok && row < M) H[((size_t)row * C + c) * N + col] = h;
          hsq[q] += h * h;
        }
    }
    rowsum_scatter(hsq, lane);
    float *g = gs + c * WN * BM;
    if constexpr (MB == 1) {
      const int q = (lane & 31) >> 1;
      if ((lane & 1) == 0) g[wn * BM + wm * TM + acc_row(q, kg)] = hsq[0];
    } else {
#pragma unroll
      for (int j = 0; j < MB / 2; ++j) {
        const int q = j + (MB / 2) * (lane & 31);
        g[wn * BM + wm * TM + (q >> 4) * 32 + acc_row(q & 15, kg)] = hsq[j];
      }
    }
  }
  __syncthreads();
  const size_t MO = (size_t)M * C;
  for (int i = tid; i < BM * C; i += NT) {
    const int t = i % BM, c = i / BM;
    const int row = m0 + t;
    if (row < M) {
      float g = 0.f;
#pragma unroll
      for (int w = 0; w < WN; ++w) g += gs[(c * WN + w) * BM + t];
      gpart[(size_t)tn * MO + (size_t)row * C + c] = g;
    }
  }
}

// ---------------------------------------------------------------------------
// Loss rows: g_r, c_r = 2 dL/dg_r, and per-block partial sums of the Eq. 1
// terms (positives and negatives apart) over 64-row blocks, one wave per block;
// the weight-gradient kernel finishes the scalar.  Each row's partials are
// summed in column-tile order, eight loads in flight.
// ---------------------------------------------------------------------------
constexpr int kLossRows = 64;

__global__ __launch_bounds__(kLossRows) void k_loss_rows(const float *__restrict__ gpart, int nt,
                                                          int R, int n_pos, float theta,
                                                          float *__restrict__ g,
                                                          float *__restrict__ c,
                                                          float *__restrict__ lpart,
                                                          float *__restrict__ s_out,
                                                          float norm_eps,
                                                          const float *__restrict__ s_in,
                                                          float *__restrict__ cs) {
  const int r = blockIdx.x * kLossRows + threadIdx.x;
  float lp = 0.f, ln = 0.f;
  if (r < R) {
    float gv = 0.f;
    int t = 0;
    for (; t + 8 <= nt; t += 8) {
      float p[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) p[j] = gpart[(size_t)(t + j) * R + r];
#pragma unroll
      for (int j = 0; j < 8; ++j) gv += p[j];
    }
    for (; t < nt; ++t) gv += gpart[(size_t)t * R + r];
    if (g) g[r] = gv;
    if (s_out) s_out[r] = 1.f / (sqrtf(gv) + norm_eps);  // g is the row's squared norm
    float cr;
    if (r < n_pos) {
      const float x = theta - gv;
      lp = softplus_f(x);
      cr = -2.f * sigmoid_f(x) / (float)n_pos;
    } else {
      const float x = gv - theta;
      ln = softplus_f(x);
      cr = 2.f * sigmoid_f(x) / (float)(R - n_pos);
    }
    c[r] = cr;
    if (cs) cs[r] = cr * s_in[r];
  }
  lp = wave_sum(lp);
  ln = wave_sum(ln);
  if (threadIdx.x == 0) {
    lpart[2 * blockIdx.x] = lp;
    lpart[2 * blockIdx.x + 1] = ln;
  }
}

// ---------------------------------------------------------------------------
// dW = (c.H)^T X_hat (+ db) with the Adam update fused.  M = d_out, N = d_in,
// K = R batch rows.  Both operands arrive row-major over K (batch rows), so the
// LDS tiles are [BK][BM] and [BK][BN].  WM x WN waves, each (BM/WM) x (BN/WN)
// as MB x NB 32x32 blocks.  A lane reads MB consecutive floats of the c.H tile
// per k and feeds one to each row block, so MFMA row i of block mb is wave-tile
// row MB*i + mb; likewise NB consecutive X_hat floats give column NB*j + nb.
// Half-wave kg takes slab rows 2s+kg.  The loads are issued raw ahead of the
// MFMAs; the row scale c, the k-tail mask and the db sums are applied when the
// registers are written to LDS.  With BS the X rows are raw (x_hat_k =
// s_k * X_k): a per-row factor of the contraction can sit on either operand,
// so the c.H rows are staged scaled by cs_k = c_k * s_k (one factor, computed
// with c by the loss kernel), the X tile is staged as loaded, and only the
// column-tile-0 workgroups, which also sum db = sum_k c_k H_k, load c.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, int PF, bool BS>
__global__ __launch_bounds__(WM *WN * 64) void k_dw_adam_f32(
    const float *__restrict__ Hm, const float *__restrict__ cvec, const float *__restrict__ Xh,
    const float *__restrict__ csvec, int M, int N, int K, float *__restrict__ W, float *__restrict__ mW, float *__restrict__ vW,
    uint16_t *__restrict__ Wb, float *__restrict__ bvec, float *__restrict__ mbv,
    float *__restrict__ vbv, AdamArgs ad, LossFinish lf) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  constexpr int LDM = BM + 4, LDN = BN + 4;
  constexpr int CFA = BM / 4, CFB = BN / 4;          // float4 per tile row
  constexpr int KSA = NT / CFA, KSB = NT / CFB;      // slab rows between a thread's loads
  constexpr int LDA = BK / KSA, LDB = BK / KSB;      // loads per thread
  static_assert(MB * 32 == TM && NB * 32 == TN, "wave tile is whole 32x32 blocks");
  static_assert(LDA * KSA == BK && LDB * KSB == BK && NT % CFA == 0 && NT % CFB == 0,
                "tile/threads");
  __shared__ __attribute__((aligned(16))) float sm[2 * BK * (LDM + LDN)];
  float *As = sm;                  // [2][BK][LDM]
  float *Bs = sm + 2 * BK * LDM;   // [2][BK][LDN]

  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;
  const bool do_db = (tn == 0);

  if (lf.loss && blockIdx.x == 0 && tid == 0) {
    float sp = 0.f, sn = 0.f;
    for (int i = 0; i < lf.nblk; ++i) {
      sp += lf.lpart[2 * i];
      sn += lf.lpart[2 * i + 1];
    }
    lf.loss[0] = sp / (float)lf.n_pos + sn / (float)lf.n_neg;
  }

  const int ca = (tid % CFA) * 4, ka = tid / CFA;
  const int cb = (tid % CFB) * 4, kb = tid / CFB;
  const float *pa = Hm + (m0 + ca < M ? m0 + ca : 0);  // invalid columns: results never stored
  const float *pb = Xh + (n0 + cb < N ? n0 + cb : 0);

  struct Stage {
    float4 a[LDA], b[LDB];
    float c[LDA], d[BS ? LDA : 1];  // product factor (c or cs); c for db under BS
    int kt;
  } st[PF];
  float4 dbp = make_float4(0.f, 0.f, 0.f, 0.f);
  auto gload = [&](Stage &g, int kt) {
#pragma unroll
    for (int i = 0; i < LDA; ++i) {
      const int k = min(kt * BK + ka + i * KSA, K - 1);
      g.a[i] = ld4(pa + (size_t)k * M);
      if constexpr (BS) {
        g.c[i] = csvec[k];
        if (do_db) g.d[i] = cvec[k];
      } else {
        g.c[i] = cvec[k];
      }
    }
#pragma unroll
    for (int i = 0; i < LDB; ++i) {
      const int k = min(kt * BK + kb + i * KSB, K - 1);
      g.b[i] = ld4(pb + (size_t)k * N);
    }
    g.kt = kt;
  };
  auto sstore = [&](const Stage &g, int buf) {
#pragma unroll
    for (int i = 0; i < LDA; ++i) {
      const bool kok = g.kt * BK + ka + i * KSA < K;  // rows past K add nothing
      const float cc = kok ? g.c[i] : 0.f;
      const float4 a = g.a[i];
      const float4 v = make_float4(a.x * cc, a.y * cc, a.z * cc, a.w * cc);
      if (do_db) {
        const float cd = BS ? (kok ? g.d[BS ? i : 0] : 0.f) : cc;
        dbp.x += a.x * cd;
        dbp.y += a.y * cd;
        dbp.z += a.z * cd;
        dbp.w += a.w * cd;
      }
      st4(As + (buf * BK + ka + i * KSA) * LDM + ca, v);
    }
#pragma unroll
    for (int i = 0; i < LDB; ++i) st4(Bs + (buf * BK + kb + i * KSB) * LDN + cb, g.b[i]);
  };

  floatx16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  auto compute = [&](int buf) {
    const float *a0 = As + (buf * BK + kg) * LDM + wm * TM + MB * li;
    const float *b0 = Bs + (buf * BK + kg) * LDN + wn * TN + NB * li;
#pragma unroll
    for (int s = 0; s < BK / 2; ++s) {
      float a[MB], b[NB];
      lds_vec<MB>(a0 + 2 * s * LDM, a);
      lds_vec<NB>(b0 + 2 * s * LDN, b);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[mb], b[nb], acc[mb][nb], 0, 0, 0);
    }
  };

  kloop<PF>((K + BK - 1) / BK, gload, sstore, compute, st);

  // Adam on this workgroup's W tile.
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = n0 + wn * TN + NB * li + nb;
    if (col >= N) continue;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * TM + MB * acc_row(r, kg) + mb;
        if (row >= M) continue;
        const size_t idx = (size_t)row * N + col;
        float p = W[idx], m = mW[idx], v = vW[idx];
        adam_update(p, m, v, acc[mb][nb][r], ad);
        W[idx] = p;
        mW[idx] = m;
        vW[idx] = v;
        if (Wb) Wb[idx] = bf16_of(p);
      }
  }

  // db and Adam on b (column-tile 0 only).
  if (do_db) {
    float *red = sm;  // [KSA][BM]
    st4(red + ka * BM + ca, dbp);
    __syncthreads();
    for (int t = tid; t < BM; t += NT) {
      const int row = m0 + t;
      if (row >= M) continue;
      float sum = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < KSA; ++g2) sum += red[g2 * BM + t];
      float p = bvec[row], m = mbv[row], v = vbv[row];
      adam_update(p, m, v, sum, ad);
      bvec[row] = p;
      mbv[row] = m;
      vbv[row] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 weight gradient as an NT product.  The contraction runs over the batch
// rows, so both operands are wanted row-major over the rows: dZ^T [d_out][Rp]
// and x_hat^T [d_in][Rp], Rp = R rounded up to 64 with zero columns.  Two
// passes write them; the product then runs on the four-wave main loop.
// ---------------------------------------------------------------------------
constexpr int kTRows = 64;  // batch rows per transposed block

// The transposes below stage a 64 x 64 bf16 tile in LDS as words of two
// consecutive rows of one column, T[col][row pair] with 33 words per column:
// the writes of a wave (one column word per lane) then fall on 64 distinct
// banks, and a lane gathers its 16 rows of a column as 8 words.
constexpr int kTWords = kTRows / 2 + 1;
// 64-column sub-tiles per workgroup of the loss pass with the bf16 operand:
// one (2048 x 2000: 8.4-8.6 against 9.3-9.7 us with two; 4096 x 3072 the same).
constexpr int kLossTSubs = 1;

// Writes rows r0..r0+63 of column `col` of a transposed tile from T (lane
// segment seg: rows 16 seg .. 16 seg + 15) to out[col][r0 + ...] (row stride Rp).
__device__ __forceinline__ void store_tcol(const uint32_t (*T)[kTWords], int c, int seg,
                                           uint16_t *out_col) {
  uint32_t w[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) w[j] = T[c][seg * 8 + j];
  uint4 *dst = reinterpret_cast<uint4 *>(out_col + seg * 16);
  dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
  dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
}

// One 64 x 64 tile of x^T [d][Rp] from bf16 rows x [R][d] (d a multiple of 8,
// zero columns R..Rp-1) through the LDS words T: the tile of rows r0.. and
// columns c0..  A lane loads eight columns of two consecutive rows.
__device__ __forceinline__ void transpose_tile(const uint16_t *__restrict__ x, int R, int Rp,
                                               int d, uint16_t *__restrict__ xT, int r0, int c0,
                                               uint32_t (*T)[kTWords]) {
  const int tid = threadIdx.x;
  {
    const int pp = tid >> 3, o = tid & 7, col = c0 + 8 * o;
    uint4 a = make_uint4(0, 0, 0, 0), b = a;
    if (col < d) {
      if (r0 + 2 * pp < R) a = ld16(x + (size_t)(r0 + 2 * pp) * d + col);
      if (r0 + 2 * pp + 1 < R) b = ld16(x + (size_t)(r0 + 2 * pp + 1) * d + col);
    }
    const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {  // columns 8o + 2j (low halves) and 8o + 2j + 1 (high)
      T[8 * o + 2 * j][pp] = (av[j] & 0xFFFFu) | (bv[j] << 16);
      T[8 * o + 2 * j + 1][pp] = (av[j] >> 16) | (bv[j] & 0xFFFF0000u);
    }
  }
  __syncthreads();
  const int c = tid >> 2, seg = tid & 3;
  if (c0 + c < d) store_tcol(T, c, seg, xT + (size_t)(c0 + c) * Rp + r0);
}

// Loss rows (as k_loss_rows, over 64-row blocks) and dZ^T = bf16(c . H)^T
// (R3) with the per-block column sums of c . H in fp32 for db:
//   grid (Rp / 64, ceil(D / (64 SUBS))); each workgroup takes 64 rows and
//   SUBS 64-column sub-tiles, staged through LDS to transpose.  The H loads of
//   all its sub-tiles are issued beside the goodness partials, before the row
//   coefficients c are known.  Every workgroup sums its rows' goodness; column
//   block 0 also writes g, c and the loss partials lpart[2 * block].
// Rows R..Rp-1 give zero columns of dZ^T.
// NEXT: the pass also writes the next layer's bf16 operand from the same H
// (pre-update activities): its rows xn [R][D] = bf16(h_r / (sqrt(g_r) + eps))
// (g_r = ||h_r||^2, the goodness) and their transpose xnT [D][Rp] (zero
// columns past R), so the next layer needs no normalisation or transpose pass.
// x (optional): the layer's bf16 input rows [R][dx]; the workgroups past the
// ny loss column blocks write their transpose xT [dx][Rp] (transpose_tile), the
// other operand of the weight-gradient product, in the same launch.
template <int SUBS, bool NEXT>
__global__ __launch_bounds__(kBlock) void k_loss_t(const float *__restrict__ gpart, int nt, int R,
                                                   int Rp, int n_pos, float theta,
                                                   const float *__restrict__ H, int D,
                                                   float *__restrict__ g_out,
                                                   float *__restrict__ c_out,
                                                   float *__restrict__ lpart,
                                                   uint16_t *__restrict__ dzT,
                                                   float *__restrict__ dbp, float norm_eps,
                                                   uint16_t *__restrict__ xn,
                                                   uint16_t *__restrict__ xnT,
                                                   const uint16_t *__restrict__ x, int dx,
                                                   uint16_t *__restrict__ xT, int ny) {
  __shared__ float cs[kTRows];
  __shared__ float ns[NEXT ? kTRows : 1];
  __shared__ float red[SUBS][16][kTRows + 4];
  __shared__ uint32_t T[SUBS][kTRows][kTWords];
  __shared__ uint32_t TN[NEXT ? SUBS : 1][kTRows][kTWords];
  const int tid = threadIdx.x;
  const int r0 = blockIdx.x * kTRows, cb0 = blockIdx.y * 64 * SUBS;
  if ((int)blockIdx.y >= ny) {  // a tile of the input's transpose (uniform per workgroup)
    transpose_tile(x, R, Rp, dx, xT, r0, (blockIdx.y - ny) * 64, T[0]);
    return;
  }
  const int q = tid & 15, p = tid >> 4;  // column quad; row pairs p and p + 16
  // rows 2p, 2p+1, 2p+32, 2p+33 of each sub-tile's column quad
  float4 v[SUBS][4];
#pragma unroll
  for (int sub = 0; sub < SUBS; ++sub)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 2 * p + (i & 1) + 32 * (i >> 1), r = r0 + row;
      const int col = cb0 + sub * 64 + 4 * q;
      v[sub][i] = (r < R && col < D) ? ld4(H + (size_t)r * D + col)
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  if (tid < kTRows) {  // wave 0: the block's rows
    const int r = r0 + tid;
    float cr = 0.f, lp = 0.f, ln = 0.f;
    if (r < R) {
      float gv = 0.f;
      int t = 0;
      for (; t + 8 <= nt; t += 8) {
        float pt[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) pt[j] = gpart[(size_t)(t + j) * R + r];
#pragma unroll
        for (int j = 0; j < 8; ++j) gv += pt[j];
      }
      for (; t < nt; ++t) gv += gpart[(size_t)t * R + r];
      if (r < n_pos) {
        const float x = theta - gv;
        lp = softplus_f(x);
        cr = -2.f * sigmoid_f(x) / (float)n_pos;
      } else {
        const float x = gv - theta;
        ln = softplus_f(x);
        cr = 2.f * sigmoid_f(x) / (float)(R - n_pos);
      }
      if (blockIdx.y == 0) {
        if (g_out) g_out[r] = gv;
        if (c_out) c_out[r] = cr;
      }
      if (NEXT) ns[tid] = 1.f / (sqrtf(gv) + norm_eps);
    } else if (NEXT) {
      ns[tid] = 0.f;
    }
    cs[tid] = cr;
    lp = wave_sum(lp);
    ln = wave_sum(ln);
    if (blockIdx.y == 0 && tid == 0) {
      lpart[2 * blockIdx.x] = lp;
      lpart[2 * blockIdx.x + 1] = ln;
    }
  }
  __syncthreads();
  float cc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) cc[i] = cs[2 * p + (i & 1) + 32 * (i >> 1)];
  if constexpr (NEXT) {  // the next layer's operand, from the unscaled activities
    float sn[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) sn[i] = ns[2 * p + (i & 1) + 32 * (i >> 1)];
#pragma unroll
    for (int sub = 0; sub < SUBS; ++sub) {
      float4 t[4];
      const int col = cb0 + sub * 64 + 4 * q;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 w = v[sub][i];
        t[i] = make_float4(w.x * sn[i], w.y * sn[i], w.z * sn[i], w.w * sn[i]);
        const int r = r0 + 2 * p + (i & 1) + 32 * (i >> 1);
        if (r < R && col < D) {
          uint2 pk;
          pk.x = pack_bf16(t[i].x, t[i].y);
          pk.y = pack_bf16(t[i].z, t[i].w);
          *reinterpret_cast<uint2 *>(xn + (size_t)r * D + col) = pk;
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float4 a = t[2 * h], b = t[2 * h + 1];
        TN[sub][4 * q + 0][p + 16 * h] = pack_bf16(a.x, b.x);
        TN[sub][4 * q + 1][p + 16 * h] = pack_bf16(a.y, b.y);
        TN[sub][4 * q + 2][p + 16 * h] = pack_bf16(a.z, b.z);
        TN[sub][4 * q + 3][p + 16 * h] = pack_bf16(a.w, b.w);
      }
    }
  }
#pragma unroll
  for (int sub = 0; sub < SUBS; ++sub) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float4 &w = v[sub][i];
      w = make_float4(w.x * cc[i], w.y * cc[i], w.z * cc[i], w.w * cc[i]);
      acc.x += w.x;
      acc.y += w.y;
      acc.z += w.z;
      acc.w += w.w;
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // the word of rows (2p, 2p+1) + 32 h of each column
      const float4 a = v[sub][2 * h], b = v[sub][2 * h + 1];
      T[sub][4 * q + 0][p + 16 * h] = pack_bf16(a.x, b.x);
      T[sub][4 * q + 1][p + 16 * h] = pack_bf16(a.y, b.y);
      T[sub][4 * q + 2][p + 16 * h] = pack_bf16(a.z, b.z);
      T[sub][4 * q + 3][p + 16 * h] = pack_bf16(a.w, b.w);
    }
    red[sub][p][4 * q + 0] = acc.x;
    red[sub][p][4 * q + 1] = acc.y;
    red[sub][p][4 * q + 2] = acc.z;
    red[sub][p][4 * q + 3] = acc.w;
  }
  __syncthreads();
  // db partials: thread (sub, column) sums its column's 16 row-group sums
  for (int i = tid; i < SUBS * 64; i += kBlock) {
    const int sub = i >> 6, c = i & 63, col = cb0 + sub * 64 + c;
    if (col < D) {
      float sum = 0.f;
#pragma unroll
      for (int k = 0; k < 16; ++k) sum += red[sub][k][c];
      dbp[(size_t)blockIdx.x * D + col] = sum;
    }
  }
  const int c = tid >> 2, seg = tid & 3;
#pragma unroll
  for (int sub = 0; sub < SUBS; ++sub) {
    const int col = cb0 + sub * 64 + c;
    if (col < D) {
      store_tcol(T[sub], c, seg, dzT + (size_t)col * Rp + r0);
      if constexpr (NEXT) store_tcol(TN[sub], c, seg, xnT + (size_t)col * Rp + r0);
    }
  }
}

typedef short i16x4 __attribute__((ext_vector_type(4)));

// gfx950 LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane j receives element j % 4 of the 8 bytes addressed by lane
// 4e + j / 4 as its element e (e = 0..3): when lane s of the group addresses
// row k0 + s / 4, columns c0 + 4 (s % 4) .. +3 of a row-major b16 tile, lane j
// gets column c0 + j at rows k0 .. k0 + 3.  (Lane layout measured on MI355X.)
__device__ __forceinline__ uint2 lds_read_tr(const uint16_t *p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4 *)(p));
  return __builtin_bit_cast(uint2, v);
}

// ---------------------------------------------------------------------------
// bf16 dW = bf16(c.H)^T X_hat (+ db from the fp32 c.H) with the Adam update
// fused.  M = d_out, N = d_in, K = R batch rows; H fp32 [K][M], X_hat bf16
// [K][N], both row-major over the contraction index.  Both LDS tiles keep that
// natural layout ([BK][BM] and [BK][BN], rows padded to 16 banks mod 64):
// staging is a coalesced copy, with H rows scaled by c in fp32 (db summed
// there) and rounded to bf16 (R3).  The MFMA fragments, eight k-consecutive
// values per lane, come from two transposed LDS reads each.  The accumulators
// go through an LDS tile so that the fused Adam reads and writes W and its
// moments with float4 accesses.
// ---------------------------------------------------------------------------
template <int BM, int BN, int BK, int WM, int WN, int PF>
__global__ __launch_bounds__(WM *WN * 64) void k_dw_adam_bf16(
    const float *__restrict__ Hm, const float *__restrict__ cvec,
    const uint16_t *__restrict__ Xh, int M, int N, int K, float *__restrict__ W,
    float *__restrict__ mW, float *__restrict__ vW, uint16_t *__restrict__ Wb,
    float *__restrict__ bvec, float *__restrict__ mbv, float *__restrict__ vbv, AdamArgs ad,
    LossFinish lf) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  constexpr int LDA = BM + 32, LDB = BN + 32;  // row strides (bf16): 16 banks mod 64
  constexpr int CA = BM / 4, CB = BN / 8;      // float4 (A) / 8-bf16 (B) chunks per row
  constexpr int RA = NT / CA, RB = NT / CB;    // slab rows between a thread's chunks
  constexpr int APT = BK / RA, BPT = BK / RB;
  static_assert(MB * 32 == TM && NB * 32 == TN, "wave tile");
  static_assert(APT * RA == BK && BPT * RB == BK && NT % CA == 0 && NT % CB == 0, "staging");
  static_assert(BK % 16 == 0, "k16 steps");
  constexpr int LDC = BN + 4;  // fp32 accumulator tile for the epilogue
  constexpr int kMain = 2 * BK * (LDA + LDB), kEpi = 2 * BM * LDC;  // in bf16 elements
  __shared__ __attribute__((aligned(16))) uint16_t sm[kMain > kEpi ? kMain : kEpi];
  uint16_t *As = sm;                 // [2][BK][LDA]
  uint16_t *Bs = sm + 2 * BK * LDA;  // [2][BK][LDB]

  const int nt = (N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, (M + BM - 1) / BM, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int li = lane & 31, kg = lane >> 5;
  const bool do_db = (tn == 0);

  if (lf.loss && blockIdx.x == 0 && tid == 0) {
    float sp = 0.f, sn = 0.f;
    for (int i = 0; i < lf.nblk; ++i) {
      sp += lf.lpart[2 * i];
      sn += lf.lpart[2 * i + 1];
    }
    lf.loss[0] = sp / (float)lf.n_pos + sn / (float)lf.n_neg;
  }

  const int ca = tid % CA, ra = tid / CA;
  const int cb = tid % CB, rb = tid / CB;
  const float *pa = Hm + min(m0 + 4 * ca, M - 4);
  const uint16_t *pb = Xh + min(n0 + 8 * cb, N - 8);

  struct Stage {
    float4 a[APT];
    float c[APT];
    uint4 b[BPT];
    int kt;
  } st[PF];
  float4 dbp = make_float4(0.f, 0.f, 0.f, 0.f);
  auto gload = [&](Stage &g, int kt) {
#pragma unroll
    for (int i = 0; i < APT; ++i) {
      const int k = min(kt * BK + ra + i * RA, K - 1);
      g.a[i] = ld4(pa + (size_t)k * M);
      g.c[i] = cvec[k];
    }
#pragma unroll
    for (int i = 0; i < BPT; ++i)
      g.b[i] = ld16(pb + (size_t)min(kt * BK + rb + i * RB, K - 1) * N);
    g.kt = kt;
  };
  auto sstore = [&](const Stage &g, int buf) {
#pragma unroll
    for (int i = 0; i < APT; ++i) {
      const int r = ra + i * RA;
      const float cc = g.kt * BK + r < K ? g.c[i] : 0.f;  // rows past K add nothing
      float4 v = g.a[i];
      v.x *= cc;
      v.y *= cc;
      v.z *= cc;
      v.w *= cc;
      if (do_db) {
        dbp.x += v.x;
        dbp.y += v.y;
        dbp.z += v.z;
        dbp.w += v.w;
      }
      uint2 p;
      p.x = pack_bf16(v.x, v.y);
      p.y = pack_bf16(v.z, v.w);
      *reinterpret_cast<uint2 *>(As + (buf * BK + r) * LDA + 4 * ca) = p;
    }
#pragma unroll
    for (int i = 0; i < BPT; ++i) st16(Bs + (buf * BK + rb + i * RB) * LDB + 8 * cb, g.b[i]);
  };

  floatx16 acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mb][nb][r] = 0.f;

  // Transposed fragment reads: within each 16-lane group g of the wave, lane
  // s reads row 8*(g/2) + 4*t + s/4 of the k16 step, columns 16*(g%2) + 4*(s%4)
  // .. +3 of the 32-wide block; the transpose hands lane (g, j) the values of
  // column 16*(g%2) + j at 4 consecutive k.  Two reads (t = 0, 1) give the 8
  // k-consecutive values v_mfma_f32_32x32x16_bf16 takes per lane.
  const int g4 = lane >> 4, s16 = lane & 15;
  const int frow = 8 * (g4 >> 1) + (s16 >> 2);
  const int fcol = 16 * (g4 & 1) + 4 * (s16 & 3);
  auto compute = [&](int buf) {
    const uint16_t *a0 = As + (buf * BK + frow) * LDA + wm * TM + fcol;
    const uint16_t *b0 = Bs + (buf * BK + frow) * LDB + wn * TN + fcol;
#pragma unroll
    for (int k16 = 0; k16 < BK; k16 += 16) {
      uint4 a[MB], b[NB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const uint2 lo = lds_read_tr(a0 + k16 * LDA + mb * 32);
        const uint2 hi = lds_read_tr(a0 + (k16 + 4) * LDA + mb * 32);
        a[mb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const uint2 lo = lds_read_tr(b0 + k16 * LDB + nb * 32);
        const uint2 hi = lds_read_tr(b0 + (k16 + 4) * LDB + nb * 32);
        b[nb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf8(a[mb]), as_bf8(b[nb]),
                                                                acc[mb][nb], 0, 0, 0);
    }
  };

  kloop<PF>((K + BK - 1) / BK, gload, sstore, compute, st);

  // Accumulators to an LDS tile in natural order, then Adam with float4
  // accesses along d_in (the main-loop buffers are free after the last barrier).
  float *Cs = reinterpret_cast<float *>(sm);  // [BM][LDC]
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        Cs[(wm * TM + mb * 32 + acc_row(r, kg)) * LDC + wn * TN + nb * 32 + li] = acc[mb][nb][r];
  __syncthreads();
  for (int idx = tid; idx < BM * (BN / 4); idx += NT) {
    const int m = idx / (BN / 4), n4 = (idx % (BN / 4)) * 4;
    const int row = m0 + m, col = n0 + n4;
    if (row >= M || col >= N) continue;
    const size_t o = (size_t)row * N + col;
    const float4 g4 = ld4(Cs + m * LDC + n4);
    float4 p = ld4(W + o), m4 = ld4(mW + o), v4 = ld4(vW + o);
    adam_update(p.x, m4.x, v4.x, g4.x, ad);
    adam_update(p.y, m4.y, v4.y, g4.y, ad);
    adam_update(p.z, m4.z, v4.z, g4.z, ad);
    adam_update(p.w, m4.w, v4.w, g4.w, ad);
    st4(W + o, p);
    st4(mW + o, m4);
    st4(vW + o, v4);
    if (Wb) {
      uint2 sh;
      sh.x = pack_bf16(p.x, p.y);
      sh.y = pack_bf16(p.z, p.w);
      *reinterpret_cast<uint2 *>(Wb + o) = sh;
    }
  }

  if (do_db) {
    __syncthreads();  // Cs reads are done
    float *red = reinterpret_cast<float *>(sm);  // [RA][BM]
    st4(red + ra * BM + 4 * ca, dbp);
    __syncthreads();
    for (int t = tid; t < BM; t += NT) {
      const int row = m0 + t;
      if (row >= M) continue;
      float sum = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < RA; ++g2) sum += red[g2 * BM + t];
      float p = bvec[row], m = mbv[row], v = vbv[row];
      adam_update(p, m, v, sum, ad);
      bvec[row] = p;
      mbv[row] = m;
      vbv[row] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Softmax prediction layer (Sec. 3 "Prediction": Softmax).  Its 10 outputs
// are far too few for MFMA tiles; the work is reading the feature rows once.
// ---------------------------------------------------------------------------
// Feature block and column of feature index f (blocks are contiguous).
__device__ __forceinline__ int head_block(const HeadFeatures &hf, int f, int &j) {
  int blk = 0, off = 0;
  while (blk + 1 < hf.n_blocks && f >= off + hf.d[blk]) off += hf.d[blk++];
  j = f - off;
  return blk;
}

// One wave per kHeadRows rows: the C dot products of each row over its
// feature blocks, reduced across the wave, then the softmax on lanes 0..C-1.
// Lanes run over features, 4 each, so a chunk is 256 consecutive features of
// one block; the chunks of all blocks form one sequence.  Each wave keeps the
// loads of the next two chunks in flight while it works on one: three
// register sets for the feature rows (the loop is unrolled by three, so each
// set is a fixed set of registers) and three LDS stages for the classifier
// weights, which go from global memory straight into LDS (buffer_load ...
// lds), C x 256 features per chunk shared by the workgroup's 4 waves, with
// one barrier per chunk.  Every chunk step issues the same loads, past the
// last chunk too (weights out of range, reading zeros; feature rows of the
// last chunk again), so the wait counts are fixed.  Rows past n are computed
// on row n-1 and never stored.  A row's sums run in the same order whatever
// its wave.
//
// CC is a compile-time bound on the class count C (C <= CC): classes C..CC-1
// load class C-1 again and their sums are dropped, so the loops have no
// per-class branches.
constexpr int kHeadRows = 2;
template <int CC>
__global__ __launch_bounds__(kBlock) void k_head_logits(HeadFeatures hf, int n, int C,
                                                        const int32_t *__restrict__ labels,
                                                        float *__restrict__ logits,
                                                        int32_t *__restrict__ pred,
                                                        float *__restrict__ G,
                                                        float *__restrict__ lrow) {
  constexpr int RW = kHeadRows, NWV = kBlock / 64, NS = 3;
  // weight loads per wave per chunk, the same for every wave: the loads past
  // slot CC-1 write slot CC-1 again, with the bytes its own load writes there
  constexpr int WL = (CC + NWV - 1) / NWV;
  constexpr int NV = WL + RW;  // vector-memory operations per wave per chunk
  static_assert(NV < 64, "wait count");
  static_assert(kHeadMaxBlocks * RW <= 64, "one lane per row scale");
  // one LDS array per stage: the compiler then sees that the weight loads
  // into one stage do not alias the reads of another, and does not wait for
  // them before those reads
  __shared__ float4 wsh0[CC * 64], wsh1[CC * 64], wsh2[CC * 64];
  __shared__ float srow[NWV][kHeadMaxBlocks][RW];
  auto stage = [&](auto S) -> float4 * {
    constexpr int s = decltype(S)::value;
    return s == 0 ? wsh0 : (s == 1 ? wsh1 : wsh2);
  };
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform, in scalar registers
  const int r0 = (blockIdx.x * NWV + wave) * RW;
  const bool active = r0 < n;  // uniform per wave; every wave stages weights
  int ng = 0;
  for (int b = 0; b < hf.n_blocks; ++b) ng += (hf.d[b] / 4 + 63) / 64;
  if (lane < hf.n_blocks * RW) {  // the rows' scale of each block
    const int b = lane / RW, r = min(r0 + lane % RW, n - 1);
    srow[wave][b][lane % RW] = hf.s[b] ? hf.s[b][r] : 1.f;
  }
  float acc[RW][CC];
#pragma unroll
  for (int q = 0; q < RW; ++q)
#pragma unroll
    for (int c = 0; c < CC; ++c) acc[q][c] = 0.f;

  // chunk cursors (block, chunk within it); the load cursor stops at the last
  // chunk, whose feature rows the steps past the end load again
  int lb = 0, lc = 0, cb = 0, cc = 0, lg = 0;
  auto next = [&](int &b, int &c) {
    if (++c == (hf.d[b] / 4 + 63) / 64) {
      ++b;
      c = 0;
    }
  };
  float4 a[NS][RW];
  auto issue = [&](auto S) {
    constexpr int s = decltype(S)::value;
    const bool past = lg >= ng;
    const int d4 = hf.d[lb] >> 2, j = lc * 64 + lane;
    const __amdgpu_buffer_rsrc_t rw =
        buffer_rsrc(hf.w[lb], (uint32_t)(((C - 1) * hf.ldw[lb] + hf.d[lb]) * 4));
#pragma unroll
    for (int i = 0; i < WL; ++i) {
      const int slot = min(i * NWV + wave, CC - 1);
      const uint32_t o = !past && j < d4
                             ? (uint32_t)((min(slot, C - 1) * hf.ldw[lb] + 4 * j) * 4)
                             : kOutOfRange;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void *)(stage(S) + slot * 64), 16, o, 0, 0, 0);
    }
    const float *h = hf.h[lb] + 4 * min(j, d4 - 1);
#pragma unroll
    for (int q = 0; q < RW; ++q) a[s][q] = ld4(h + (size_t)min(r0 + q, n - 1) * hf.d[lb]);
    ++lg;
    if (lg < ng) next(lb, lc);
  };
  auto compute = [&](auto S) {
    constexpr int s = decltype(S)::value;
    const int d4 = hf.d[cb] >> 2, j = cc * 64 + lane;
    if (active && j < d4) {
      float4 x[RW];
#pragma unroll
      for (int q = 0; q < RW; ++q) {
        const float sr = srow[wave][cb][q];
        x[q] = a[s][q];
        x[q].x *= sr;
        x[q].y *= sr;
        x[q].z *= sr;
        x[q].w *= sr;
      }
#pragma unroll
      for (int c = 0; c < CC; ++c) {
        const float4 w = stage(S)[c * 64 + lane];
#pragma unroll
        for (int q = 0; q < RW; ++q)
          acc[q][c] += x[q].x * w.x + x[q].y * w.y + x[q].z * w.z + x[q].w * w.w;
      }
    }
    next(cb, cc);
  };
  // Step g: chunk g's loads have landed (only chunk g+1's may be in flight)
  // and, past the barrier, every wave has them and is done with stage g-1,
  // which chunk g+2's weights then refill.
  auto step = [&](auto S, int g) {
    constexpr int s = decltype(S)::value;
    __builtin_amdgcn_s_waitcnt(vmcnt_wait(NV));
    lds_barrier();
    issue(std::integral_constant<int, (s + 2) % NS>{});
    if (g < ng) compute(S);
  };
  issue(std::integral_constant<int, 0>{});
  issue(std::integral_constant<int, 1>{});
  for (int g = 0; g < ng; g += NS) {
    step(std::integral_constant<int, 0>{}, g);
    step(std::integral_constant<int, 1>{}, g + 1);
    step(std::integral_constant<int, 2>{}, g + 2);
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_wait(0));  // no weight load outlives the loop
  if (!active) return;
#pragma unroll
  for (int q = 0; q < RW; ++q) {
    const int r = r0 + q;
    if (r >= n) break;  // uniform per wave
    float z = 0.f, zmax = -INFINITY;
    int arg = 0;
#pragma unroll
    for (int c = 0; c < CC; ++c)
      if (c < C) {
        float v = wave_sum(acc[q][c]);
        for (int k = 0; k < hf.n_bias; ++k) v += hf.bias[k][c];
        if (lane == c) z = v;
        if (v > zmax) {
          zmax = v;
          arg = c;
        }
      }
    const float e = lane < C ? expf(z - zmax) : 0.f;
    const float esum = wave_sum(e);
    // labels outside [0, C) are clamped into it (unspecified result, no stray access)
    const int y = labels ? min(max(labels[r], 0), C - 1) : 0;
    const float zy = __shfl(z, y);  // the true class's logit, from its lane (whole wave active)
    if (lane < C) {
      if (logits) logits[(size_t)r * C + lane] = z;
      if (G) G[(size_t)r * C + lane] = (e / esum - (lane == y ? 1.f : 0.f)) / (float)n;
    }
    if (lane == 0) {
      if (pred) pred[r] = arg;
      if (lrow) lrow[r] = logf(esum) - (zy - zmax);  // -log p_y
    }
  }
}

// Backprop of a layer's classifier into the layer: one thread per 4
// consecutive units of a row.
template <int CC>  // class-count bound, as in k_head_logits
__global__ __launch_bounds__(kBlock) void k_po_dz(const float *__restrict__ H,
                                                  const float *__restrict__ G,
                                                  const float *__restrict__ Wc, int R, int D,
                                                  int C, float *__restrict__ dZ,
                                                  float *__restrict__ ones) {
  const int q = blockIdx.x * kBlock + threadIdx.x;
  const int d4 = D >> 2;
  if (q >= R * d4) return;
  const int r = q / d4, j = 4 * (q % d4);
  const float4 h = ld4(H + (size_t)r * D + j);
  float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int c = 0; c < CC; ++c) {
    const int cc = min(c, C - 1);
    const float gl = G[(size_t)r * C + cc];
    const float4 w = ld4(Wc + (size_t)cc * D + j);
    const float gc = c < C ? gl : 0.f;
    g.x += gc * w.x;
    g.y += gc * w.y;
    g.z += gc * w.z;
    g.w += gc * w.w;
  }
  g.x = h.x > 0.f ? g.x : 0.f;  // the ReLU derivative (h = 0 wherever z <= 0)
  g.y = h.y > 0.f ? g.y : 0.f;
  g.z = h.z > 0.f ? g.z : 0.f;
  g.w = h.w > 0.f ? g.w : 0.f;
  st4(dZ + (size_t)r * D + j, g);
  if (j == 0) ones[r] = 1.f;
}

// Classifier weight-gradient partials.  A workgroup covers 64 consecutive
// features (16 float4 lanes) of one split of rows, with 16 row lanes walking
// the split's rows 16 apart; each thread keeps C float4 sums, and the 16 row
// lanes are reduced through LDS in a fixed order.  A split of 128 rows leaves
// each thread 8 independent row loads, and a 1024-row step of 2000 features
// has 256 workgroups (one thread per feature quad and split had left 16
// workgroups walking 128 dependent rows each).
constexpr int kHeadGradQuads = 16, kHeadGradRowLanes = kBlock / kHeadGradQuads;
template <int CC>  // class-count bound, as in k_head_logits
__global__ __launch_bounds__(kBlock) void k_head_grad(HeadFeatures hf,
                                                      const float *__restrict__ G, int n, int C,
                                                      int D, int rows_per_split,
                                                      float *__restrict__ part) {
  __shared__ float4 red[kHeadGradRowLanes][CC][kHeadGradQuads];
  const int q = threadIdx.x % kHeadGradQuads, rl = threadIdx.x / kHeadGradQuads;
  const int f = 4 * (blockIdx.x * kHeadGradQuads + q);
  const bool fok = f < D;
  int j = 0;
  const int blk = fok ? head_block(hf, f, j) : 0;
  const int d = hf.d[blk];
  const float *h = hf.h[blk] + j;
  const float *sv = hf.s[blk];  // null: scale 1
  const int r0 = blockIdx.y * rows_per_split, r1 = min(n, r0 + rows_per_split);
  float4 acc[CC];
#pragma unroll
  for (int c = 0; c < CC; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (fok) {
    for (int r = r0 + rl; r < r1; r += kHeadGradRowLanes) {
      float4 a = ld4(h + (size_t)r * d);
      const float sr = sv ? sv[r] : 1.f;
      a.x *= sr;
      a.y *= sr;
      a.z *= sr;
      a.w *= sr;
#pragma unroll
      for (int c = 0; c < CC; ++c) {
        const float g = G[(size_t)r * C + min(c, C - 1)];  // classes past C: never stored
        acc[c].x += g * a.x;
        acc[c].y += g * a.y;
        acc[c].z += g * a.z;
        acc[c].w += g * a.w;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < CC; ++c) red[rl][c][q] = acc[c];
  __syncthreads();
  for (int o = threadIdx.x; o < CC * kHeadGradQuads; o += kBlock) {
    const int c = o / kHeadGradQuads, qq = o % kHeadGradQuads;
    const int ff = 4 * (blockIdx.x * kHeadGradQuads + qq);
    if (c >= C || ff >= D) continue;
    float4 sum = red[0][c][qq];
    for (int k = 1; k < kHeadGradRowLanes; ++k) {
      const float4 v = red[k][c][qq];
      sum.x += v.x;
      sum.y += v.y;
      sum.z += v.z;
      sum.w += v.w;
    }
    st4(part + ((size_t)blockIdx.y * C + c) * D + ff, sum);
  }
}

// Adam on the head.  Block 0 also reduces db and the loss over the rows: each
// thread sums a fixed strided subset, then a fixed-order tree in LDS.
__global__ __launch_bounds__(kBlock) void k_head_adam(const float *__restrict__ part, int splits,
                                                      const float *__restrict__ G,
                                                      const float *__restrict__ lrow, int n,
                                                      int C, int D, float *__restrict__ W,
                                                      float *__restrict__ mW,
                                                      float *__restrict__ vW,
                                                      float *__restrict__ bvec,
                                                      float *__restrict__ mbv,
                                                      float *__restrict__ vbv, AdamArgs ad,
                                                      float *__restrict__ loss) {
  const size_t i = 4 * ((size_t)blockIdx.x * kBlock + threadIdx.x);
  const size_t total = (size_t)C * D;
  if (i < total) {
    float4 g = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < splits; ++sp) {
      const float4 v = ld4(part + (size_t)sp * total + i);
      g.x += v.x;
      g.y += v.y;
      g.z += v.z;
      g.w += v.w;
    }
    float4 p = ld4(W + i), m = ld4(mW + i), v = ld4(vW + i);
    adam_update(p.x, m.x, v.x, g.x, ad);
    adam_update(p.y, m.y, v.y, g.y, ad);
    adam_update(p.z, m.z, v.z, g.z, ad);
    adam_update(p.w, m.w, v.w, g.w, ad);
    st4(W + i, p);
    st4(mW + i, m);
    st4(vW + i, v);
  }
  if (blockIdx.x != 0) return;
  __shared__ float red[kHeadMaxClasses + 1][kBlock];
  float acc[kHeadMaxClasses + 1];
#pragma unroll
  for (int c = 0; c <= kHeadMaxClasses; ++c) acc[c] = 0.f;
  for (int r = threadIdx.x; r < n; r += kBlock) {
#pragma unroll
    for (int c = 0; c < kHeadMaxClasses; ++c)
      if (c < C) acc[c] += G[(size_t)r * C + c];
    if (lrow) acc[kHeadMaxClasses] += lrow[r];
  }
#pragma unroll
  for (int c = 0; c <= kHeadMaxClasses; ++c) red[c][threadIdx.x] = acc[c];
  __syncthreads();
  for (int st = kBlock / 2; st > 0; st >>= 1) {
    if ((int)threadIdx.x < st)
#pragma unroll
      for (int c = 0; c <= kHeadMaxClasses; ++c) red[c][threadIdx.x] += red[c][threadIdx.x + st];
    __syncthreads();
  }
  if ((int)threadIdx.x < C) {
    const int c = threadIdx.x;
    float p = bvec[c], m = mbv[c], v = vbv[c];
    adam_update(p, m, v, red[c][0], ad);
    bvec[c] = p;
    mbv[c] = m;
    vbv[c] = v;
  }
  if (threadIdx.x == 0 && loss) loss[0] = red[kHeadMaxClasses][0] / (float)n;
}

// ---------------------------------------------------------------------------
// Small kernels
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_goodness(const float *__restrict__ gpart, int nt,
                                                     int R, float *__restrict__ g,
                                                     float *__restrict__ out, int accumulate,
                                                     float *__restrict__ s_out, float norm_eps) {
  const int r = blockIdx.x * kBlock + threadIdx.x;
  if (r >= R) return;
  float gv = 0.f;
  for (int t = 0; t < nt; ++t) gv += gpart[(size_t)t * R + r];
  if (g) g[r] = gv;
  if (s_out) s_out[r] = 1.f / (sqrtf(gv) + norm_eps);
  if (out) out[r] = accumulate ? out[r] + gv : gv;
}

// pred[i] = argmax_c S[i][c], lowest c on ties.  With `exclude`, label
// exclude[i] takes no part (an out-of-range label excludes nothing); C >= 2 then.
__global__ __launch_bounds__(kBlock) void k_argmax(const float *__restrict__ S, int n, int C,
                                                   const int32_t *__restrict__ exclude,
                                                   int32_t *__restrict__ pred) {
  const int i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const float *s = S + (size_t)i * C;
  const int skip = exclude ? exclude[i] : -1;
  int arg = skip == 0 ? 1 : 0;
  float best = s[arg];
  for (int c = arg + 1; c < C; ++c)
    if (c != skip && s[c] > best) {
      best = s[c];
      arg = c;
    }
  pred[i] = arg;
}

// Eight weights per thread: two 16-byte loads, one 16-byte store.
__global__ __launch_bounds__(kBlock) void k_bf16_shadow(const float *__restrict__ W,
                                                        uint16_t *__restrict__ Wb, size_t count) {
  const size_t i = ((size_t)blockIdx.x * kBlock + threadIdx.x) * 8;
  if (i + 8 <= count) {
    const float4 a = ld4(W + i), b = ld4(W + i + 4);
    st16(Wb + i, make_uint4(pack_bf16(a.x, a.y), pack_bf16(a.z, a.w), pack_bf16(b.x, b.y),
                            pack_bf16(b.z, b.w)));
  } else {
    for (size_t j = i; j < count; ++j) Wb[j] = bf16_of(W[j]);
  }
}

inline unsigned cdiv(long a, long b) { return (unsigned)((a + b - 1) / b); }

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
// GEMM tile configurations: (BM, BN, BK in elements, waves along M, waves
// along N, stages: register stages of a weight-gradient load pipeline, LDS
// stages of a forward one), measured on MI355X over the layer shapes of the
// workloads.  A weight-gradient launch takes the large
// tile when its tiles fill the CUs (fp32: three quarters of them), else the
// small one.
// FOUR: the bf16 forward runs on the four-wave kernel (k_fwd4) with this tile.
template <int BM, int BN, int BK, int WM, int WN, int PF = 1, bool FOUR = false>
struct Tile {
  static constexpr int bm = BM, bn = BN, bk = BK, wm = WM, wn = WN, pf = PF,
                       threads = WM * WN * 64;
  static constexpr bool four = FOUR;
  static long tiles(int m, int n) { return (long)cdiv(m, BM) * cdiv(n, BN); }
};
constexpr int kCUs = 256;
using DwBig = Tile<64, 128, 32, 2, 4, 3>;
using DwSmall = Tile<64, 64, 32, 2, 2, 2>;
using DwBigBf16 = Tile<128, 128, 32, 4, 2, 2>;
// Fewer than two bf16 tiles per CU: one more register stage (2000x2000 over
// 2048 rows 54 -> 50 us; at 3072x3072 over 4096 rows two stages are faster).
using DwFullBf16 = Tile<128, 128, 32, 4, 2, 3>;
using DwSmallBf16 = Tile<64, 64, 64, 2, 2, 2>;

// Forward tile ladder: a launch takes the largest tile whose grid still puts a
// workgroup on every CU.  The last parameter of a forward tile is its number
// of LDS stages (BK is fixed at 128 bytes of a row): two let two 128x128
// workgroups share a CU.  A bf16 k-tile holds a quarter of the MFMA time of
// an fp32 one, too little to cover a load's latency with one tile in flight,
// so a bf16 grid of fewer than two 128x128 workgroups per CU (Full) takes
// three stages instead, as does the bf16 small tile (the fp32 one measured
// faster with two: 1024x2000x2000, 88 -> 77 us).  bf16 products use the larger
// tiles for operand reuse when the grid allows: 256x192 on the four-wave
// kernel (one workgroup per CU) when its grid fills the CUs, and 256x256 on
// eight waves only from two of its tiles per CU on, where it measured faster.
// fp32 takes 128x256 on eight waves (one workgroup per CU) only from 16 of its
// tiles per CU on: 81920x2000x2000 ran 5027 us on it against 5173 us on
// 128x128, but 18080 rows (1136 such tiles, 4.4 per CU) 1238 against 1108 us.
// The fp32 128x128 tile runs on 16 waves (32x32 each, four per SIMD): alone,
// 2048x2000x2000 130 against 135 us on 8 waves, the label-expanding layer 0
// of scoring 319 against 336 us; the epochs measured the same.
template <bool BF16>
struct FwdTiles;
template <>
struct FwdTiles<false> {
  using Huge = Tile<128, 256, 32, 2, 4, 2>;
  using Large = Tile<128, 128, 32, 4, 4, 2>;
  using Big = Large;
  using Full = Large;
  using Small = Tile<64, 64, 32, 2, 2, 2>;
};
template <>
struct FwdTiles<true> {
  using Huge = Tile<256, 256, 64, 4, 2, 2>;
  using Large = Tile<256, 192, 64, 2, 2, 2, true>;  // four-wave kernel (k_fwd4)
  using Big = Tile<128, 128, 64, 4, 2, 2>;
  using Full = Tile<128, 128, 64, 4, 2, 3>;
  using Small = Tile<64, 64, 64, 2, 2, 3>;
};
template <class T>
struct TileTag {
  using type = T;
};
// LARGE = false: the label-expanding forward, whose epilogue holds more per
// row, stays on the 128x128 / 64x64 rungs.
template <bool BF16, bool LARGE = true, class F>
void fwd_tile(int M, int N, F &&f) {
  using L = FwdTiles<BF16>;
  if constexpr (LARGE) {
    if (L::Huge::tiles(M, N) >= (BF16 ? 2 : 16) * kCUs) return f(TileTag<typename L::Huge>{});
    if (L::Large::tiles(M, N) >= kCUs) return f(TileTag<typename L::Large>{});
  }
  if (L::Big::tiles(M, N) >= 2 * kCUs) return f(TileTag<typename L::Big>{});
  if (L::Full::tiles(M, N) >= kCUs) return f(TileTag<typename L::Full>{});
  f(TileTag<typename L::Small>{});
}

// The fp32 large tile also takes grids of at least three quarters of the CUs:
// layer 0's 2000x784 weights (224 tiles) ran 91 us on it over 2048 rows,
// 98 us on 416 small tiles.
inline bool dw_big(int M, int N, int dtype) {
  return dtype ? DwBigBf16::tiles(M, N) >= kCUs : 4 * DwBig::tiles(M, N) >= 3 * kCUs;
}

int fwd_col_tiles(int rows, int n_cols, int dtype) {
  int bn = 0;
  auto pick = [&](auto t) { bn = decltype(t)::type::bn; };
  if (dtype)
    fwd_tile<true>(rows, n_cols, pick);
  else
    fwd_tile<false>(rows, n_cols, pick);
  return (int)cdiv(n_cols, bn);
}
int fwd_expand_col_tiles(int rows, int n_cols, int dtype) {
  int bn = 0;
  auto pick = [&](auto t) { bn = decltype(t)::type::bn; };
  if (dtype)
    fwd_tile<true, false>(rows, n_cols, pick);
  else
    fwd_tile<false, false>(rows, n_cols, pick);
  return (int)cdiv(n_cols, bn);
}
int fwd_col_tiles_max(int n_cols) {
  return (int)cdiv(n_cols, std::min(FwdTiles<false>::Small::bn, FwdTiles<true>::Small::bn));
}

int loss_blocks(int rows) { return (int)cdiv(rows, kLossRows); }
static_assert(kLossRows == kTRows, "the two loss kernels share their row blocks");
int padded_rows(int rows) { return (int)cdiv(rows, kTRows) * kTRows; }

template <int NV>
void embed_norm_reg(const RowMap &m, int rows, int d, float eps, bool normalise, bool bf16_out,
                    void *out, float *scale_out, hipStream_t s) {
  const dim3 grid(cdiv(rows, kBlock / 64));
  if (bf16_out)
    hipLaunchKernelGGL((k_embed_norm_reg<NV, true>), grid, dim3(kBlock), 0, s, m, rows, d, eps,
                       (int)normalise, out, scale_out);
  else
    hipLaunchKernelGGL((k_embed_norm_reg<NV, false>), grid, dim3(kBlock), 0, s, m, rows, d, eps,
                       (int)normalise, out, scale_out);
}

hipError_t launch_embed_norm(const RowMap &m, int rows, int d, float eps, bool normalise,
                             bool bf16_out, void *out, float *scale_out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int nv = (int)cdiv(d / 4, 64);  // float4 per lane for the whole row
  if (nv <= 1) {
    embed_norm_reg<1>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else if (nv <= 2) {
    embed_norm_reg<2>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else if (nv <= 4) {
    embed_norm_reg<4>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else if (nv <= 8) {
    embed_norm_reg<8>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else if (nv <= 12) {
    embed_norm_reg<12>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else if (nv <= 16) {
    embed_norm_reg<16>(m, rows, d, eps, normalise, bf16_out, out, scale_out, s);
  } else {
    const dim3 grid(cdiv(rows, kBlock / 64));
    if (bf16_out)
      hipLaunchKernelGGL(k_embed_norm<true>, grid, dim3(kBlock), 0, s, m, rows, d, eps,
                         (int)normalise, out, scale_out);
    else
      hipLaunchKernelGGL(k_embed_norm<false>, grid, dim3(kBlock), 0, s, m, rows, d, eps,
                         (int)normalise, out, scale_out);
  }
  return hipGetLastError();
}

template <bool BF16, class T>
void fwd_launch(const void *x, const void *w, const float *bias, const float *rowscale, int M,
                int N, int K, float *H, float *gpart, hipStream_t s) {
  using E = typename Operand<BF16>::T;
  const dim3 grid(T::tiles(M, N));
  const E *xe = static_cast<const E *>(x);
  const E *we = static_cast<const E *>(w);
  static_assert(T::bk == nt_bk<BF16>(), "forward k-tile is 128 bytes");
  if constexpr (BF16 && T::four) {
    static_assert(T::wm == 2 && T::wn == 2, "four-wave tile");
    if (H)
      hipLaunchKernelGGL((k_fwd4<T::bm, T::bn, T::pf, true>), grid, dim3(256), 0, s, xe, we, bias,
                         rowscale, M, N, K, H, gpart);
    else
      hipLaunchKernelGGL((k_fwd4<T::bm, T::bn, T::pf, false>), grid, dim3(256), 0, s, xe, we,
                         bias, rowscale, M, N, K, H, gpart);
  } else if (H) {
    hipLaunchKernelGGL((k_fwd<BF16, T::bm, T::bn, T::wm, T::wn, T::pf, true>), grid,
                       dim3(T::threads), 0, s, xe, we, bias, rowscale, M, N, K, H, gpart);
  } else {
    hipLaunchKernelGGL((k_fwd<BF16, T::bm, T::bn, T::wm, T::wn, T::pf, false>), grid,
                       dim3(T::threads), 0, s, xe, we, bias, rowscale, M, N, K, H, gpart);
  }
}

hipError_t launch_fwd(int dtype, const void *X, const void *W, const float *bias,
                      const float *rowscale, int M, int N, int K, float *H, float *gpart,
                      hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K > kMaxWidth) return hipErrorInvalidValue;
  if (dtype == 0)
    fwd_tile<false>(M, N, [&](auto t) {
      fwd_launch<false, typename decltype(t)::type>(X, W, bias, rowscale, M, N, K, H, gpart, s);
    });
  else
    fwd_tile<true>(M, N, [&](auto t) {
      fwd_launch<true, typename decltype(t)::type>(X, W, bias, rowscale, M, N, K, H, gpart, s);
    });
  return hipGetLastError();
}

template <bool BF16, class T>
void fwd_expand_launch(const void *x, const void *w, const float *bias, const LabelExpand &ex,
                       int M, int N, int K, float *H, float *gpart, hipStream_t s) {
  using E = typename Operand<BF16>::T;
  const dim3 grid(T::tiles(M, N));
  const E *xe = static_cast<const E *>(x);
  const E *we = static_cast<const E *>(w);
  static_assert(T::bk == nt_bk<BF16>(), "forward k-tile is 128 bytes");
  if (H)
    hipLaunchKernelGGL((k_fwd_expand<BF16, T::bm, T::bn, T::wm, T::wn, T::pf, true>), grid,
                       dim3(T::threads), 0, s, xe, we, bias, ex, M, N, K, H, gpart);
  else
    hipLaunchKernelGGL((k_fwd_expand<BF16, T::bm, T::bn, T::wm, T::wn, T::pf, false>), grid,
                       dim3(T::threads), 0, s, xe, we, bias, ex, M, N, K, H, gpart);
}

hipError_t launch_fwd_expand(int dtype, const void *X, const void *W, const float *bias,
                             const LabelExpand &ex, int M, int N, int K, float *H, float *gpart,
                             hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (ex.n_classes < 1 || ex.n_classes > kMaxExpand || ex.n_classes > K || K > kMaxWidth)
    return hipErrorInvalidValue;
  if (dtype == 0)
    fwd_tile<false, false>(M, N, [&](auto t) {
      fwd_expand_launch<false, typename decltype(t)::type>(X, W, bias, ex, M, N, K, H, gpart, s);
    });
  else
    fwd_tile<true, false>(M, N, [&](auto t) {
      fwd_expand_launch<true, typename decltype(t)::type>(X, W, bias, ex, M, N, K, H, gpart, s);
    });
  return hipGetLastError();
}

hipError_t launch_loss(const float *gpart, int ntiles, int R, int n_pos, float theta, float *g,
                       float *c, float *lpart, float *s_out, float norm_eps, const float *s_in,
                       float *cs, hipStream_t s) {
  if (cs && !s_in) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_loss_rows, dim3(loss_blocks(R)), dim3(kLossRows), 0, s, gpart, ntiles, R,
                     n_pos, theta, g, c, lpart, s_out, norm_eps, s_in, cs);
  return hipGetLastError();
}

hipError_t launch_loss_t(const float *gpart, int ntiles, int R, int n_pos, float theta,
                        const float *H, int D, float *g, float *c, float *lpart, uint16_t *dzT,
                        float *dbp, float norm_eps, uint16_t *xn, uint16_t *xnT,
                        const uint16_t *x, int dx, uint16_t *xT, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (D % 4 || (xn == nullptr) != (xnT == nullptr) || (x == nullptr) != (xT == nullptr) ||
      (x && dx % 8))
    return hipErrorInvalidValue;
  const int Rp = padded_rows(R);
  constexpr int subs = kLossTSubs;
  const int ny = (int)cdiv(D, 64 * subs);
  const dim3 grid(Rp / kTRows, ny + (x ? (int)cdiv(dx, 64) : 0));
  if (xn)
    hipLaunchKernelGGL((k_loss_t<subs, true>), grid, dim3(kBlock), 0, s, gpart, ntiles, R, Rp,
                       n_pos, theta, H, D, g, c, lpart, dzT, dbp, norm_eps, xn, xnT, x, dx, xT,
                       ny);
  else
    hipLaunchKernelGGL((k_loss_t<subs, false>), grid, dim3(kBlock), 0, s, gpart, ntiles, R, Rp,
                       n_pos, theta, H, D, g, c, lpart, dzT, dbp, norm_eps, xn, xnT, x, dx, xT,
                       ny);
  return hipGetLastError();
}

// The bf16 weight-gradient product takes 192x192 tiles when they give every CU
// one (3072-wide layers), else 128x128 with four LDS stages (2000x2000 over
// 2048 rows: 36.3 against 37.1 us with three).
template <int BM, int BN, int NBUF>
void dw4_launch(const uint16_t *dzT, const uint16_t *xT, int M, int N, int K, float *G, float *W,
                float *mW, float *vW, uint16_t *Wb, const float *dbp, int nrb, float *b, float *mb,
                float *vb, const AdamArgs &a, const LossFinish &lf, hipStream_t s) {
  const dim3 grid(cdiv(M, BM) * cdiv(N, BN));
  if (G)
    hipLaunchKernelGGL((k_dw4<BM, BN, NBUF, false>), grid, dim3(256), 0, s, dzT, xT, M, N, K, G,
                       W, mW, vW, Wb, dbp, nrb, b, mb, vb, a, lf);
  else
    hipLaunchKernelGGL((k_dw4<BM, BN, NBUF, true>), grid, dim3(256), 0, s, dzT, xT, M, N, K, G, W,
                       mW, vW, Wb, dbp, nrb, b, mb, vb, a, lf);
}

bool dw4_split_adam(int M, int N) { return (long)cdiv(M, 192) * cdiv(N, 192) >= kCUs; }

hipError_t launch_dw4(const uint16_t *dzT, const uint16_t *xT, int M, int N, int R, float *G,
                      float *W, float *mW, float *vW, uint16_t *Wb, const float *dbp, float *b,
                      float *mb, float *vb, const AdamArgs &a, const LossFinish &lf,
                      hipStream_t s) {
  const int Rp = padded_rows(R), nrb = Rp / kTRows;
  if (N % 8 || Rp > kMaxWidth) return hipErrorInvalidValue;
  if (dw4_split_adam(M, N))  // the 192x192 rung: one tile per CU
    dw4_launch<192, 192, 3>(dzT, xT, M, N, Rp, G, W, mW, vW, Wb, dbp, nrb, b, mb, vb, a, lf, s);
  else
    dw4_launch<128, 128, 4>(dzT, xT, M, N, Rp, G, W, mW, vW, Wb, dbp, nrb, b, mb, vb, a, lf, s);
  return hipGetLastError();
}

hipError_t launch_adam_dense(const float *G, int M, int N, float *W, float *mW, float *vW,
                             uint16_t *Wb, const float *dbp, int R, float *b, float *mb,
                             float *vb, const AdamArgs &a, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (N % 4) return hipErrorInvalidValue;
  const int nrb = padded_rows(R) / kTRows;
  const int nmain = (int)cdiv((long)M * N / 4, (long)kBlock * kAdamDenseBatch);
  const int nbias = (int)cdiv(M, kBlock);
  hipLaunchKernelGGL(k_adam_dense, dim3(nmain + nbias), dim3(kBlock), 0, s, G, M, N, nmain, W, mW,
                     vW, Wb, dbp, nrb, b, mb, vb, a);
  return hipGetLastError();
}

template <bool BF16, class T>
void dw_launch(const float *H, const float *c, const void *Xh, const float *cs, int M, int N,
               int K, float *W, float *mW, float *vW, uint16_t *Wb, float *b, float *mb,
               float *vb, const AdamArgs &a, const LossFinish &lf, hipStream_t s) {
  const dim3 grid(T::tiles(M, N)), block(T::threads);
  if constexpr (BF16)
    hipLaunchKernelGGL((k_dw_adam_bf16<T::bm, T::bn, T::bk, T::wm, T::wn, T::pf>), grid, block,
                       0, s, H, c, static_cast<const uint16_t *>(Xh), M, N, K, W, mW, vW, Wb, b,
                       mb, vb, a, lf);
  else if (cs)
    hipLaunchKernelGGL((k_dw_adam_f32<T::bm, T::bn, T::bk, T::wm, T::wn, T::pf, true>), grid,
                       block, 0, s, H, c, static_cast<const float *>(Xh), cs, M, N, K, W, mW,
                       vW, Wb, b, mb, vb, a, lf);
  else
    hipLaunchKernelGGL((k_dw_adam_f32<T::bm, T::bn, T::bk, T::wm, T::wn, T::pf, false>), grid,
                       block, 0, s, H, c, static_cast<const float *>(Xh), cs, M, N, K, W, mW,
                       vW, Wb, b, mb, vb, a, lf);
}

hipError_t launch_dw_adam(int dtype, const float *H, const float *c, const void *Xh,
                          const float *cs, int M, int N, int K, float *W, float *mW,
                          float *vW, uint16_t *Wb, float *b, float *mb, float *vb,
                          const AdamArgs &a, const LossFinish &lf, hipStream_t s) {
  const bool big = dw_big(M, N, dtype);
  if (dtype == 0) {
    if (big)
      dw_launch<false, DwBig>(H, c, Xh, cs, M, N, K, W, mW, vW, Wb, b, mb, vb, a, lf, s);
    else
      dw_launch<false, DwSmall>(H, c, Xh, cs, M, N, K, W, mW, vW, Wb, b, mb, vb, a, lf, s);
  } else {
    if (cs) return hipErrorInvalidValue;  // bf16 operands arrive normalised
    if (big && DwBigBf16::tiles(M, N) >= 2 * kCUs)
      dw_launch<true, DwBigBf16>(H, c, Xh, nullptr, M, N, K, W, mW, vW, Wb, b, mb, vb, a, lf, s);
    else if (big)
      dw_launch<true, DwFullBf16>(H, c, Xh, nullptr, M, N, K, W, mW, vW, Wb, b, mb, vb, a, lf, s);
    else
      dw_launch<true, DwSmallBf16>(H, c, Xh, nullptr, M, N, K, W, mW, vW, Wb, b, mb, vb, a, lf,
                                   s);
  }
  return hipGetLastError();
}

hipError_t launch_goodness(const float *gpart, int ntiles, int R, float *g, float *out,
                           int accumulate, float *s_out, float norm_eps, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_goodness, dim3(cdiv(R, kBlock)), dim3(kBlock), 0, s, gpart, ntiles, R, g,
                     out, accumulate, s_out, norm_eps);
  return hipGetLastError();
}

hipError_t launch_argmax(const float *scores, int n, int C, const int32_t *exclude, int32_t *pred,
                         hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_argmax, dim3(cdiv(n, kBlock)), dim3(kBlock), 0, s, scores, n, C, exclude,
                     pred);
  return hipGetLastError();
}

// Calls f with the compile-time class-count bound of the head kernels for C.
template <class F>
void head_classes(int C, F &&f) {
  static_assert(kHeadMaxClasses == 16, "bounds below");
  if (C <= 2) return f(std::integral_constant<int, 2>{});
  if (C <= 4) return f(std::integral_constant<int, 4>{});
  if (C <= 8) return f(std::integral_constant<int, 8>{});
  if (C <= 10) return f(std::integral_constant<int, 10>{});
  f(std::integral_constant<int, 16>{});
}

hipError_t launch_head_logits(const HeadFeatures &f, int n, int C, const int32_t *labels,
                              float *logits, int32_t *pred, float *G, float *lrow,
                              hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (C < 1 || C > kHeadMaxClasses || f.n_blocks < 1 || f.n_blocks > kHeadMaxBlocks ||
      f.n_bias < 0 || f.n_bias > kHeadMaxBlocks || ((G || lrow) && !labels))
    return hipErrorInvalidValue;
  for (int b = 0; b < f.n_blocks; ++b)  // whole float4 of features; weight offsets in 32 bits
    if (f.d[b] <= 0 || f.d[b] % 4 || f.ldw[b] < f.d[b] ||
        ((long)(C - 1) * f.ldw[b] + f.d[b]) * 4 >= (1l << 31))
      return hipErrorInvalidValue;
  head_classes(C, [&](auto cc) {
    hipLaunchKernelGGL(k_head_logits<decltype(cc)::value>, dim3(cdiv(n, kBlock / 64 * kHeadRows)),
                       dim3(kBlock), 0, s, f, n, C, labels, logits, pred, G, lrow);
  });
  return hipGetLastError();
}

hipError_t launch_po_dz(const float *H, const float *G, const float *Wc, int R, int D, int C,
                        float *dZ, float *ones, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (C < 1 || C > kHeadMaxClasses || D % 4) return hipErrorInvalidValue;
  head_classes(C, [&](auto cc) {
    hipLaunchKernelGGL(k_po_dz<decltype(cc)::value>, dim3(cdiv((long)R * (D / 4), kBlock)),
                       dim3(kBlock), 0, s, H, G, Wc, R, D, C, dZ, ones);
  });
  return hipGetLastError();
}

int head_grad_splits(int n) { return std::max(1, (int)cdiv(n, 128)); }

hipError_t launch_head_grad(const HeadFeatures &f, const float *G, int n, int C, int D,
                            int splits, float *part, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (C < 1 || C > kHeadMaxClasses || D % 4 || splits < 1) return hipErrorInvalidValue;
  const int rps = (int)cdiv(n, splits);
  head_classes(C, [&](auto cc) {
    hipLaunchKernelGGL(k_head_grad<decltype(cc)::value>,
                       dim3(cdiv(D / 4, kHeadGradQuads), splits), dim3(kBlock), 0, s, f, G, n, C,
                       D, rps, part);
  });
  return hipGetLastError();
}

hipError_t launch_head_adam(const float *part, int splits, const float *G, const float *lrow,
                            int n, int C, int D, float *W, float *mW, float *vW, float *b,
                            float *mb, float *vb, const AdamArgs &a, float *loss,
                            hipStream_t s) {
  if (C < 1 || C > kHeadMaxClasses || D % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_head_adam, dim3(std::max(1u, cdiv((long)C * D / 4, kBlock))),
                     dim3(kBlock), 0, s, part, splits, G, lrow, n, C, D, W, mW, vW, b, mb, vb,
                     a, loss);
  return hipGetLastError();
}

hipError_t launch_bf16_shadow(const float *W, uint16_t *Wb, size_t count, hipStream_t s) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(k_bf16_shadow, dim3(cdiv((long)count, 8 * kBlock)), dim3(kBlock), 0, s, W,
                     Wb, count);
  return hipGetLastError();
}

}  // namespace ffk
