// gfx950 (CDNA4) kernels of the Forward-Forward training step and label scoring.
//
// Method: Aktemur et al., "Going Forward-Forward in Distributed Deep Learning"
// (arXiv 2404.08573), Sec. 3 (goodness, Eq. 1; prediction), Sec. 5.1 (layers, Adam).
//
// Kernels
//   k_embed_norm   label embedding (Sec. 3 "Negative Data") + row L2 normalisation;
//                  one wave per row, float4 loads, HBM-bound.
//   k_fwd_f32      Z = X W^T on fp32 MFMA (v_mfma_f32_32x32x2f32), epilogue fuses
//                  bias, ReLU, the H store and the per-row goodness partial sum over
//                  the tile's columns (Eq. 1) through a lane butterfly and LDS.
//   k_loss         goodness partials -> g, the Eq. 1 threshold loss and the per-row
//                  gradient coefficient c_r = 2 dL/dg_r; one workgroup, fixed order.
//   k_dw_adam_f32  dW = (c.H)^T X_hat on fp32 MFMA (contraction over the batch rows),
//                  the row scale c applied while staging H, db summed from the same
//                  staged rows, and the Adam update of W and b fused in the epilogue
//                  (no split over rows, so every dW tile is final in one workgroup).
//   k_goodness, k_argmax, k_bf16_shadow: small row/elementwise kernels.
//
// Every reduction runs in a fixed order, so results are bitwise reproducible
// run to run and independent of stream interleaving.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ff_internal.h"

namespace ffk {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBlock = 256;  // 4 waves of 64 lanes

__device__ __forceinline__ float4 ld4(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}
__device__ __forceinline__ void st4(float *p, float4 v) { *reinterpret_cast<float4 *>(p) = v; }
__device__ __forceinline__ float comp(const float4 &v, int q) {
  return q == 0 ? v.x : (q == 1 ? v.y : (q == 2 ? v.z : v.w));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float softplus_f(float x) {
  return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x)));
}
__device__ __forceinline__ float sigmoid_f(float x) {
  const float e = expf(-fabsf(x));
  return x >= 0.f ? 1.f / (1.f + e) : e / (1.f + e);
}

__device__ __forceinline__ void adam_update(float &p, float &m, float &v, float g,
                                            const AdamArgs &a) {
  m = a.beta1 * m + (1.f - a.beta1) * g;
  v = a.beta2 * v + (1.f - a.beta2) * g * g;
  const float mh = m / a.bc1;
  const float vh = v / a.bc2;
  p = p - a.lr * mh / (sqrtf(vh) + a.eps);
}

// ---------------------------------------------------------------------------
// Row source mapping (label embedding) + L2 normalisation
// ---------------------------------------------------------------------------
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
  } else {
    src = r;
    lab = -1;
  }
}

__device__ __forceinline__ float4 embed4(float4 v, int col, int lab, int C) {
  if (lab >= 0 && col < C) {
    v.x = (col + 0 == lab) ? 1.f : (col + 0 < C ? 0.f : v.x);
    v.y = (col + 1 == lab) ? 1.f : (col + 1 < C ? 0.f : v.y);
    v.z = (col + 2 == lab) ? 1.f : (col + 2 < C ? 0.f : v.z);
    v.w = (col + 3 == lab) ? 1.f : (col + 3 < C ? 0.f : v.w);
  }
  return v;
}

template <bool BF16OUT>
__global__ __launch_bounds__(kBlock) void k_embed_norm(RowMap m, int rows, int d, float eps,
                                                       int normalise, void *out) {
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
    scale = 1.f / (sqrtf(ss) + eps);
  }
  for (int i = lane; i < d4; i += 64) {
    float4 v = embed4(ld4(xr + 4 * i), 4 * i, lab, m.n_classes);
    v.x *= scale;
    v.y *= scale;
    v.z *= scale;
    v.w *= scale;
    if (BF16OUT) {
      uint2 p;
      p.x = bf16_bits(v.x) | (bf16_bits(v.y) << 16);
      p.y = bf16_bits(v.z) | (bf16_bits(v.w) << 16);
      reinterpret_cast<uint2 *>(out)[(size_t)r * d4 + i] = p;
    } else {
      st4(reinterpret_cast<float *>(out) + (size_t)r * d + 4 * i, v);
    }
  }
}

// ---------------------------------------------------------------------------
// Goodness row reduction of a 64x64 wave tile held as 2x2 32x32 MFMA blocks.
// v[q], q = bi*16 + r, holds this lane's partial (over its columns) for the
// accumulator row (bi, r).  A reduce-scatter butterfly over the 32 lanes of
// each half-wave leaves lane l with the full sum of entry q = l & 31.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float rowsum_scatter32(float (&v)[32], int lane) {
#pragma unroll
  for (int o = 16, half = 16; o >= 1; o >>= 1, half >>= 1) {
    const bool hi = (lane & o) != 0;
#pragma unroll
    for (int q = 0; q < half; ++q) {
      const float send = hi ? v[q] : v[q + half];
      const float keep = hi ? v[q + half] : v[q];
      v[q] = keep + __shfl_xor(send, o);
    }
  }
  return v[0];
}

// Row (within the wave's 64-row tile) of 32x32 accumulator element (bi, r)
// held by a lane with half-wave index kg: the v_mfma_f32_32x32x2f32 output
// layout puts row 8*(r/4) + 4*kg + r%4 of block bi in register r.
__device__ __forceinline__ int acc_row(int bi, int r, int kg) {
  return bi * 32 + 8 * (r >> 2) + 4 * kg + (r & 3);
}

// ---------------------------------------------------------------------------
// Forward: H = relu(X W^T + b), gpart[tn][row] = sum over the tile's columns of H^2.
// X [M][K], W [N][K] (both K-contiguous), fp32.  Tile 128x128, 4 waves in 2x2,
// each wave 64x64 as 2x2 blocks of v_mfma_f32_32x32x2f32.  Within a BK slab the
// two half-waves take the two halves of the slab's k range, so every lane reads
// contiguous float4 runs from LDS for both operands (the k order inside the
// contraction is a permutation of the plain order, the same for X and W).
// ---------------------------------------------------------------------------
template <int BK, bool STORE_H>
__global__ __launch_bounds__(kBlock) void k_fwd_f32(const float *__restrict__ X,
                                                    const float *__restrict__ W,
                                                    const float *__restrict__ bias, int M, int N,
                                                    int K, float *__restrict__ H,
                                                    float *__restrict__ gpart) {
  constexpr int BM = 128, BN = 128;
  constexpr int LDK = BK + 4;   // padded row: conflict-free 16-byte reads
  constexpr int KF4 = BK / 4;   // float4 per tile row
  constexpr int A_LD = BM * KF4 / kBlock;
  constexpr int B_LD = BN * KF4 / kBlock;
  static_assert(A_LD * kBlock == BM * KF4 && B_LD * kBlock == BN * KF4, "tile/threads");
  __shared__ __attribute__((aligned(16))) float sm[2 * (BM + BN) * LDK];
  float *As = sm;                 // [2][BM][LDK]
  float *Bs = sm + 2 * BM * LDK;  // [2][BN][LDK]

  const int nt = (N + BN - 1) / BN;
  const int tn = blockIdx.x % nt, tm = blockIdx.x / nt;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, kg = lane >> 5;

  float4 ra[A_LD], rb[B_LD];
  auto gload = [&](int kt) {
    const int kb = kt * BK;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int idx = tid + i * kBlock, row = idx / KF4, kc = (idx % KF4) * 4;
      const int gr = m0 + row, gk = kb + kc;
      ra[i] = (gr < M && gk < K) ? ld4(X + (size_t)gr * K + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + i * kBlock, row = idx / KF4, kc = (idx % KF4) * 4;
      const int gr = n0 + row, gk = kb + kc;
      rb[i] = (gr < N && gk < K) ? ld4(W + (size_t)gr * K + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int idx = tid + i * kBlock, row = idx / KF4, kc = (idx % KF4) * 4;
      st4(As + (buf * BM + row) * LDK + kc, ra[i]);
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + i * kBlock, row = idx / KF4, kc = (idx % KF4) * 4;
      st4(Bs + (buf * BN + row) * LDK + kc, rb[i]);
    }
  };

  floatx16 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  auto compute = [&](int buf) {
    const float *a0 = As + (buf * BM + wm * 64 + li) * LDK + kg * (BK / 2);
    const float *b0 = Bs + (buf * BN + wn * 64 + li) * LDK + kg * (BK / 2);
#pragma unroll
    for (int s4 = 0; s4 < BK / 2; s4 += 4) {
      float4 a[2], b[2];
      a[0] = ld4(a0 + s4);
      a[1] = ld4(a0 + 32 * LDK + s4);
      b[0] = ld4(b0 + s4);
      b[1] = ld4(b0 + 32 * LDK + s4);
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
          for (int bj = 0; bj < 2; ++bj)
            acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(comp(a[bi], q), comp(b[bj], q),
                                                               acc[bi][bj], 0, 0, 0);
    }
  };

  const int nk = (K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    compute(cur);
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: bias, ReLU, H store, goodness partials.
  float hsq[32];
#pragma unroll
  for (int q = 0; q < 32; ++q) hsq[q] = 0.f;
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    const int col = n0 + wn * 64 + bj * 32 + li;
    const bool cok = col < N;
    const float bv = cok ? bias[col] : 0.f;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float h = cok ? fmaxf(acc[bi][bj][r] + bv, 0.f) : 0.f;
        if (STORE_H) {
          const int row = m0 + wm * 64 + acc_row(bi, r, kg);
          if (row < M && cok) H[(size_t)row * N + col] = h;
        }
        hsq[bi * 16 + r] += h * h;
      }
  }
  const float part = rowsum_scatter32(hsq, lane);
  const int q = lane & 31;
  float *gs = sm;  // [2][BM], main-loop buffers are free after the last barrier
  gs[wn * BM + wm * 64 + acc_row(q >> 4, q & 15, kg)] = part;
  __syncthreads();
  if (tid < BM) {
    const int row = m0 + tid;
    if (row < M) gpart[(size_t)tn * M + row] = gs[tid] + gs[BM + tid];
  }
}

// ---------------------------------------------------------------------------
// Loss: one workgroup; g_r, c_r, and the Eq. 1 loss (mean over positives +
// mean over negatives) with a fixed-order tree reduction.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_loss(const float *__restrict__ gpart, int nt, int R,
                                               int n_pos, float theta, float *__restrict__ g,
                                               float *__restrict__ c, float *__restrict__ loss) {
  __shared__ float sp[1024], sn[1024];
  const int n_neg = R - n_pos;
  const float inv_p = 1.f / (float)n_pos, inv_n = 1.f / (float)n_neg;
  float lp = 0.f, ln = 0.f;
  for (int r = threadIdx.x; r < R; r += 1024) {
    float gv = 0.f;
    for (int t = 0; t < nt; ++t) gv += gpart[(size_t)t * R + r];
    if (g) g[r] = gv;
    if (r < n_pos) {
      const float x = theta - gv;
      lp += softplus_f(x);
      c[r] = -2.f * sigmoid_f(x) * inv_p;
    } else {
      const float x = gv - theta;
      ln += softplus_f(x);
      c[r] = 2.f * sigmoid_f(x) * inv_n;
    }
  }
  sp[threadIdx.x] = lp;
  sn[threadIdx.x] = ln;
  __syncthreads();
  for (int s = 512; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) {
      sp[threadIdx.x] += sp[threadIdx.x + s];
      sn[threadIdx.x] += sn[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0 && loss) loss[0] = sp[0] * inv_p + sn[0] * inv_n;
}

// ---------------------------------------------------------------------------
// dW = (c.H)^T X_hat (+ db) with the Adam update fused.  M = d_out, N = d_in,
// K = R batch rows.  Both operands arrive row-major over K (batch rows), so the
// LDS tiles are [BK][BM] and [BK][BN]; each lane reads one float per operand
// per MFMA.  Half-wave kg takes slab rows 2s+kg; the 32-float pad puts those
// two rows on disjoint bank halves.
// ---------------------------------------------------------------------------
template <int BK>
__global__ __launch_bounds__(kBlock) void k_dw_adam_f32(
    const float *__restrict__ Hm, const float *__restrict__ cvec, const float *__restrict__ Xh,
    int M, int N, int K, float *__restrict__ W, float *__restrict__ mW, float *__restrict__ vW,
    uint16_t *__restrict__ Wb, float *__restrict__ bvec, float *__restrict__ mb,
    float *__restrict__ vb, AdamArgs ad) {
  constexpr int BM = 128, BN = 128;
  constexpr int LDM = BM + 32, LDN = BN + 32;
  constexpr int MF4 = BM / 4, NF4 = BN / 4;
  constexpr int A_LD = BK * MF4 / kBlock, B_LD = BK * NF4 / kBlock;
  constexpr int RG = kBlock / MF4;  // row groups of the staging layout
  static_assert(A_LD * kBlock == BK * MF4 && B_LD * kBlock == BK * NF4, "tile/threads");
  __shared__ __attribute__((aligned(16))) float sm[2 * BK * (LDM + LDN)];
  float *As = sm;                  // [2][BK][LDM]
  float *Bs = sm + 2 * BK * LDM;   // [2][BK][LDN]

  const int nt = (N + BN - 1) / BN;
  const int tn = blockIdx.x % nt, tm = blockIdx.x / nt;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 31, kg = lane >> 5;
  const bool do_db = (tn == 0);

  float4 ra[A_LD], rb[B_LD];
  float4 dbp = make_float4(0.f, 0.f, 0.f, 0.f);
  auto gload = [&](int kt) {
    const int kb = kt * BK;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int idx = tid + i * kBlock, k = idx / MF4, c4 = (idx % MF4) * 4;
      const int gr = kb + k, gc = m0 + c4;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (gr < K && gc < M) {
        v = ld4(Hm + (size_t)gr * M + gc);
        const float cc = cvec[gr];
        v.x *= cc;
        v.y *= cc;
        v.z *= cc;
        v.w *= cc;
      }
      ra[i] = v;
      if (do_db) {
        dbp.x += v.x;
        dbp.y += v.y;
        dbp.z += v.z;
        dbp.w += v.w;
      }
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + i * kBlock, k = idx / NF4, c4 = (idx % NF4) * 4;
      const int gr = kb + k, gc = n0 + c4;
      rb[i] = (gr < K && gc < N) ? ld4(Xh + (size_t)gr * N + gc) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int idx = tid + i * kBlock, k = idx / MF4, c4 = (idx % MF4) * 4;
      st4(As + (buf * BK + k) * LDM + c4, ra[i]);
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + i * kBlock, k = idx / NF4, c4 = (idx % NF4) * 4;
      st4(Bs + (buf * BK + k) * LDN + c4, rb[i]);
    }
  };

  floatx16 acc[2][2];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  auto compute = [&](int buf) {
    const float *a0 = As + (buf * BK + kg) * LDM + wm * 64 + li;
    const float *b0 = Bs + (buf * BK + kg) * LDN + wn * 64 + li;
#pragma unroll
    for (int s = 0; s < BK / 2; ++s) {
      const float a_0 = a0[2 * s * LDM], a_1 = a0[2 * s * LDM + 32];
      const float b_0 = b0[2 * s * LDN], b_1 = b0[2 * s * LDN + 32];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a_0, b_0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a_0, b_1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a_1, b_0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a_1, b_1, acc[1][1], 0, 0, 0);
    }
  };

  const int nk = (K + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    compute(cur);
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // Adam on this workgroup's W tile.
#pragma unroll
  for (int bj = 0; bj < 2; ++bj) {
    const int col = n0 + wn * 64 + bj * 32 + li;
    if (col >= N) continue;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + wm * 64 + acc_row(bi, r, kg);
        if (row >= M) continue;
        const size_t idx = (size_t)row * N + col;
        float p = W[idx], m = mW[idx], v = vW[idx];
        adam_update(p, m, v, acc[bi][bj][r], ad);
        W[idx] = p;
        mW[idx] = m;
        vW[idx] = v;
        if (Wb) Wb[idx] = (uint16_t)bf16_bits(p);
      }
  }

  // db and Adam on b (column-tile 0 only).
  if (do_db) {
    float *red = sm;  // [RG][BM]
    const int rg = tid / MF4, c4 = (tid % MF4) * 4;
    st4(red + rg * BM + c4, dbp);
    __syncthreads();
    if (tid < BM && m0 + tid < M) {
      float s = 0.f;
#pragma unroll
      for (int g2 = 0; g2 < RG; ++g2) s += red[g2 * BM + tid];
      const int row = m0 + tid;
      float p = bvec[row], m = mb[row], v = vb[row];
      adam_update(p, m, v, s, ad);
      bvec[row] = p;
      mb[row] = m;
      vb[row] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Small kernels
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_goodness(const float *__restrict__ gpart, int nt,
                                                     int R, float *__restrict__ g,
                                                     float *__restrict__ out, int accumulate) {
  const int r = blockIdx.x * kBlock + threadIdx.x;
  if (r >= R) return;
  float gv = 0.f;
  for (int t = 0; t < nt; ++t) gv += gpart[(size_t)t * R + r];
  if (g) g[r] = gv;
  if (out) out[r] = accumulate ? out[r] + gv : gv;
}

__global__ __launch_bounds__(kBlock) void k_argmax(const float *__restrict__ S, int n, int C,
                                                   int32_t *__restrict__ pred) {
  const int i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const float *s = S + (size_t)i * C;
  float best = s[0];
  int arg = 0;
  for (int c = 1; c < C; ++c)
    if (s[c] > best) {
      best = s[c];
      arg = c;
    }
  pred[i] = arg;
}

__global__ __launch_bounds__(kBlock) void k_bf16_shadow(const float *__restrict__ W,
                                                        uint16_t *__restrict__ Wb, size_t count) {
  const size_t i = (size_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < count) Wb[i] = (uint16_t)bf16_bits(W[i]);
}

inline unsigned cdiv(long a, long b) { return (unsigned)((a + b - 1) / b); }

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
int fwd_col_tiles(int n_cols, int /*dtype*/) { return (int)cdiv(n_cols, 128); }

hipError_t launch_embed_norm(const RowMap &m, int rows, int d, float eps, bool normalise,
                             bool bf16_out, void *out, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid(cdiv(rows, kBlock / 64));
  if (bf16_out)
    hipLaunchKernelGGL(k_embed_norm<true>, grid, dim3(kBlock), 0, s, m, rows, d, eps,
                       (int)normalise, out);
  else
    hipLaunchKernelGGL(k_embed_norm<false>, grid, dim3(kBlock), 0, s, m, rows, d, eps,
                       (int)normalise, out);
  return hipGetLastError();
}

hipError_t launch_fwd(int dtype, const void *X, const void *W, const float *bias, int M, int N,
                      int K, float *H, float *gpart, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (dtype != 0) return hipErrorNotSupported;
  const dim3 grid(cdiv(M, 128) * cdiv(N, 128));
  const float *x = static_cast<const float *>(X);
  const float *w = static_cast<const float *>(W);
  if (H)
    hipLaunchKernelGGL((k_fwd_f32<32, true>), grid, dim3(kBlock), 0, s, x, w, bias, M, N, K, H,
                       gpart);
  else
    hipLaunchKernelGGL((k_fwd_f32<32, false>), grid, dim3(kBlock), 0, s, x, w, bias, M, N, K, H,
                       gpart);
  return hipGetLastError();
}

hipError_t launch_loss(const float *gpart, int ntiles, int R, int n_pos, float theta, float *g,
                       float *c, float *loss, hipStream_t s) {
  hipLaunchKernelGGL(k_loss, dim3(1), dim3(1024), 0, s, gpart, ntiles, R, n_pos, theta, g, c,
                     loss);
  return hipGetLastError();
}

hipError_t launch_dw_adam(int dtype, const float *H, const float *c, const void *Xh, int M, int N,
                          int K, float *W, float *mW, float *vW, uint16_t *Wb, float *b, float *mb,
                          float *vb, const AdamArgs &a, hipStream_t s) {
  if (dtype != 0) return hipErrorNotSupported;
  const dim3 grid(cdiv(M, 128) * cdiv(N, 128));
  hipLaunchKernelGGL((k_dw_adam_f32<32>), grid, dim3(kBlock), 0, s, H, c,
                     static_cast<const float *>(Xh), M, N, K, W, mW, vW, Wb, b, mb, vb, a);
  return hipGetLastError();
}

hipError_t launch_goodness(const float *gpart, int ntiles, int R, float *g, float *out,
                           int accumulate, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_goodness, dim3(cdiv(R, kBlock)), dim3(kBlock), 0, s, gpart, ntiles, R, g,
                     out, accumulate);
  return hipGetLastError();
}

hipError_t launch_argmax(const float *scores, int n, int C, int32_t *pred, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_argmax, dim3(cdiv(n, kBlock)), dim3(kBlock), 0, s, scores, n, C, pred);
  return hipGetLastError();
}

hipError_t launch_bf16_shadow(const float *W, uint16_t *Wb, size_t count, hipStream_t s) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(k_bf16_shadow, dim3(cdiv((long)count, kBlock)), dim3(kBlock), 0, s, W, Wb,
                     count);
  return hipGetLastError();
}

}  // namespace ffk
