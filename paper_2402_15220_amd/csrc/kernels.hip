// gfx950 (MI355X) kernels for decode attention over a prefix-tree, chunked
// KV cache with the two-phase partition of ChunkAttention (arXiv 2402.15220,
// Section 3.2).
//
// Pools: K and V, each [slot][head][c][d]; slot_len[slot] holds the number of
// valid rows of every slot. q and o: [B][H][d] in tree row order.
// Softmax runs in base 2: scores are multiplied by scale*log2(e), so partial
// maxima stored in the workspace are in log2 units.
//
//   kcf  chunk-first phase (Algorithm 1, Eqn 1). One workgroup per (segment
//        of shared chunks, head, block of <= 16*NRT covered rows). For every
//        64-token block of a chunk it forms S^T = K Q^T on the matrix cores
//        (the covered query rows batched as the N dimension), updates the
//        online softmax per row, and accumulates O^T = V^T P^T, again on the
//        matrix cores. It writes one unnormalised partial (O, m, n) per row.
//   ksf  sequence-first phase (Algorithm 2). One workgroup per (row, head,
//        split): a bandwidth-bound pass over the row's private chunks with
//        16-byte loads, sub-wavefront DPP reductions for q.k, and per-lane
//        online softmax; then the row's chunk-first partials are folded in
//        with attn_reduce (Eqn 2) and O/n is written.
//   kmg  merge epilogue for rows whose private chunks were split over
//        several workgroups (Eqn 2 over every partial of the row, then O/n).
//   kkv  K/V row copies for tree operations (new chunks, split tails).
#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

#include "kernels.hpp"

namespace ca {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr float kNegBig = -FLT_MAX;  // "no score yet": exp2(kNegBig - x) == 0, never NaN

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over aligned groups of N lanes (N = 8, 16, 32 or 64); every lane of the
// group receives the sum. Must be called with the whole wavefront active.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror: groups of 8
  if constexpr (N >= 16) x += dpp<0x140>(x);  // row_mirror: rows of 16
  if constexpr (N >= 32) x += __shfl_xor(x, 16);
  if constexpr (N >= 64) x += __shfl_xor(x, 32);
  return x;
}

template <typename T>
struct Elem;
template <>
struct Elem<_Float16> {
  static constexpr int kPerVec = 8;  // elements per 16-byte vector
  __device__ static __forceinline__ void unpack(const uint4& r, float* f) {
    const half8 h = __builtin_bit_cast(half8, r);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = static_cast<float>(h[i]);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    half8 h;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = static_cast<_Float16>(f[i]);
    return __builtin_bit_cast(uint4, h);
  }
};
template <>
struct Elem<float> {
  static constexpr int kPerVec = 4;
  __device__ static __forceinline__ void unpack(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x);
    f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z);
    f[3] = __uint_as_float(r.w);
  }
  __device__ static __forceinline__ uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
  }
};

// attn_reduce (Eqn 2) in base 2: fold (mo, no, acco) into (m, n, acc).
template <int E>
__device__ __forceinline__ void fold(float& m, float& n, float* acc, float mo, float no,
                                     const float* acco) {
  const float mm = fmaxf(m, mo);
  const float a = fast_exp2(m - mm);
  const float b = fast_exp2(mo - mm);
  n = n * a + no * b;
#pragma unroll
  for (int j = 0; j < E; ++j) acc[j] = acc[j] * a + acco[j] * b;
  m = mm;
}

// ---------------------------------------------------------------------------
// Sequence-first phase.

struct KsfParams {
  const void* q;
  void* o;
  const void* kpool;
  const void* vpool;
  const int32_t* slot_len;
  const SfItem* items;
  const int32_t* priv_slot;
  const int32_t* part_ptr;
  const int32_t* parts;
  float* ws_o;
  float2* ws_ml;
  int H;
  int C;
  float qscale;
};

// Lane layout: a token row of d elements is read by LPT = d/EPL lanes, 16
// bytes each; a wavefront load instruction covers TPW = 64/LPT consecutive
// tokens (1 KiB), the four wavefronts cover consecutive groups of TPW tokens
// and every lane issues U such loads per step, so one step streams 64 tokens
// of K and of V of the chunk. Each group of LPT lanes keeps its own running
// (m, n, acc) over the tokens it saw; the groups are combined at the end.
template <typename T, int D>
__global__ __launch_bounds__(256) void ksf_kernel(KsfParams P) {
  using E = Elem<T>;
  constexpr int EPL = E::kPerVec;
  constexpr int LPT = D / EPL;
  constexpr int TPW = 64 / LPT;
  constexpr int TPS = TPW * 4;
  constexpr int U = 64 / TPS;
  static_assert(U >= 1 && TPS * U == 64, "step must cover 64 tokens");

  const SfItem it = P.items[blockIdx.x];
  const int h = blockIdx.y;
  const int H = P.H, C = P.C;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int sub = lane % LPT, tr = lane / LPT;

  float qf[EPL];
  {
    const uint4 qr = *reinterpret_cast<const uint4*>(static_cast<const T*>(P.q) +
                                                     (static_cast<size_t>(it.row) * H + h) * D +
                                                     sub * EPL);
    E::unpack(qr, qf);
  }

  float m = kNegBig, n = 0.f, acc[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) acc[j] = 0.f;

  const T* kpool = static_cast<const T*>(P.kpool);
  const T* vpool = static_cast<const T*>(P.vpool);
  for (int ci = it.cb; ci < it.ce; ++ci) {
    const int slot = P.priv_slot[ci];
    const int len = P.slot_len[slot];
    const size_t base = (static_cast<size_t>(slot) * H + h) * static_cast<size_t>(C) * D + sub * EPL;
    const T* kb = kpool + base;
    const T* vb = vpool + base;
    for (int t0 = 0; t0 < len; t0 += 64) {
      uint4 kr[U], vr[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int tok = t0 + u * TPS + w * TPW + tr;
        if (tok < len) {
          kr[u] = *reinterpret_cast<const uint4*>(kb + static_cast<size_t>(tok) * D);
          vr[u] = *reinterpret_cast<const uint4*>(vb + static_cast<size_t>(tok) * D);
        } else {
          kr[u] = make_uint4(0, 0, 0, 0);
          vr[u] = make_uint4(0, 0, 0, 0);
        }
      }
      float s[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float kf[EPL];
        E::unpack(kr[u], kf);
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < EPL; ++j) dot = fmaf(qf[j], kf[j], dot);
        s[u] = group_sum<LPT>(dot);
      }
      float mx = kNegBig;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int tok = t0 + u * TPS + w * TPW + tr;
        s[u] = tok < len ? s[u] * P.qscale : -INFINITY;
        mx = fmaxf(mx, s[u]);
      }
      const float mn = fmaxf(m, mx);
      const float alpha = fast_exp2(m - mn);
      n *= alpha;
#pragma unroll
      for (int j = 0; j < EPL; ++j) acc[j] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = fast_exp2(s[u] - mn);
        n += p;
        float vf[EPL];
        E::unpack(vr[u], vf);
#pragma unroll
        for (int j = 0; j < EPL; ++j) acc[j] = fmaf(p, vf[j], acc[j]);
      }
      m = mn;
    }
  }

  // combine the token-row groups of this wavefront
#pragma unroll
  for (int off = LPT; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m, off);
    const float no = __shfl_xor(n, off);
    float ao[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) ao[j] = __shfl_xor(acc[j], off);
    fold<EPL>(m, n, acc, mo, no, ao);
  }
  // combine the four wavefronts
  __shared__ float st[4][LPT][EPL + 2];
  if (tr == 0) {
    st[w][sub][0] = m;
    st[w][sub][1] = n;
#pragma unroll
    for (int j = 0; j < EPL; ++j) st[w][sub][2 + j] = acc[j];
  }
  __syncthreads();
  if (w != 0 || tr != 0) return;
#pragma unroll
  for (int ww = 1; ww < 4; ++ww) fold<EPL>(m, n, acc, st[ww][sub][0], st[ww][sub][1], &st[ww][sub][2]);

  if (it.out_part < 0) {
    // fold the chunk-first partials of this row (Algorithm 2), then O/n
    for (int k = P.part_ptr[it.row]; k < P.part_ptr[it.row + 1]; ++k) {
      const int p = P.parts[k];
      const float2 ml = P.ws_ml[static_cast<size_t>(p) * H + h];
      const float* po = P.ws_o + (static_cast<size_t>(p) * H + h) * D + sub * EPL;
      float ao[EPL];
#pragma unroll
      for (int j = 0; j < EPL; j += 4) {
        const float4 x = *reinterpret_cast<const float4*>(po + j);
        ao[j] = x.x;
        ao[j + 1] = x.y;
        ao[j + 2] = x.z;
        ao[j + 3] = x.w;
      }
      fold<EPL>(m, n, acc, ml.x, ml.y, ao);
    }
    const float inv = 1.f / n;
#pragma unroll
    for (int j = 0; j < EPL; ++j) acc[j] *= inv;
    *reinterpret_cast<uint4*>(static_cast<T*>(P.o) + (static_cast<size_t>(it.row) * H + h) * D +
                              sub * EPL) = E::pack(acc);
  } else {
    float* po = P.ws_o + (static_cast<size_t>(it.out_part) * H + h) * D + sub * EPL;
#pragma unroll
    for (int j = 0; j < EPL; j += 4)
      *reinterpret_cast<float4*>(po + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
    if (sub == 0) P.ws_ml[static_cast<size_t>(it.out_part) * H + h] = make_float2(m, n);
  }
}

// ---------------------------------------------------------------------------
// Merge epilogue for split rows.

struct KmgParams {
  void* o;
  const int32_t* mg_rows;
  const int32_t* part_ptr;
  const int32_t* parts;
  const float* ws_o;
  const float2* ws_ml;
  int H;
};

template <typename T, int D>
__global__ __launch_bounds__(64) void kmg_kernel(KmgParams P) {
  constexpr int E = D / 64;
  const int row = P.mg_rows[blockIdx.x];
  const int h = blockIdx.y, H = P.H;
  const int lane = threadIdx.x;
  float m = kNegBig, n = 0.f, acc[E];
#pragma unroll
  for (int j = 0; j < E; ++j) acc[j] = 0.f;
  for (int k = P.part_ptr[row]; k < P.part_ptr[row + 1]; ++k) {
    const int p = P.parts[k];
    const float2 ml = P.ws_ml[static_cast<size_t>(p) * H + h];
    const float* po = P.ws_o + (static_cast<size_t>(p) * H + h) * D;
    float ao[E];
#pragma unroll
    for (int j = 0; j < E; ++j) ao[j] = po[lane + 64 * j];
    fold<E>(m, n, acc, ml.x, ml.y, ao);
  }
  const float inv = 1.f / n;
  T* o = static_cast<T*>(P.o) + (static_cast<size_t>(row) * H + h) * D;
#pragma unroll
  for (int j = 0; j < E; ++j) o[lane + 64 * j] = static_cast<T>(acc[j] * inv);
}

// ---------------------------------------------------------------------------
// Chunk-first phase on the matrix cores.

struct KcfParams {
  const void* q;
  const void* kpool;
  const void* vpool;
  const int32_t* slot_len;
  const CfSeg* segs;
  const int32_t* seg_slots;
  float* ws_o;
  float2* ws_ml;
  int H;
  int C;
  float qscale;
};

// Matrix-core operand layout used below (16x16 output tiles, 64 lanes;
// l16 = lane % 16, g = lane / 16):
//   A (16 x K): lane holds row l16, its K-slice g;   B (K x 16): column l16,
//   K-slice g;   C/D (16 x 16): lane holds rows 4g..4g+3 of column l16.
// Both operands use the same K-slice per lane, so the contraction does not
// depend on how the hardware orders K inside a slice.
//
// Wavefront w owns tokens 16w..16w+15 of each 64-token block for S^T and the
// d columns [w*D/4, (w+1)*D/4) for O^T. P = exp2(S - m) travels through LDS
// (as [row][token]) and V is staged in LDS ([token][d], rows padded by two
// elements so the transposed A-operand reads of four lane groups fall in
// disjoint banks).
template <int D, int NRT>
__global__ __launch_bounds__(256) void kcf_f16_kernel(KcfParams P) {
  constexpr int KS = D / 32;  // 16x16x32 steps over d for S^T
  constexpr int DT = D / 64;  // 16-wide d tiles per wavefront for O^T
  constexpr int VS = D + 2;   // V row stride in LDS (halves)
  constexpr int PS = 64 + 8;  // P row stride in LDS (halves), keeps 16-byte row alignment
  constexpr int R = 16 * NRT;
  __shared__ _Float16 v_lds[64 * VS];
  __shared__ _Float16 p_lds[R * PS];
  __shared__ float red[4][R];

  const CfSeg sg = P.segs[blockIdx.x];
  const int h = blockIdx.y, H = P.H, C = P.C;
  const int rb = sg.row_begin + static_cast<int>(blockIdx.z) * R;
  const int nrows = min(R, sg.row_end - rb);
  if (nrows <= 0) return;
  const int nrt = (nrows + 15) / 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const _Float16* q = static_cast<const _Float16*>(P.q);
  const _Float16* kpool = static_cast<const _Float16*>(P.kpool);
  const _Float16* vpool = static_cast<const _Float16*>(P.vpool);

  half8 qf[NRT][KS];
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    const int r = 16 * t + l16;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (r < nrows)
        qf[t][s] = *reinterpret_cast<const half8*>(q + (static_cast<size_t>(rb + r) * H + h) * D +
                                                   32 * s + 8 * g);
      else
        qf[t][s] = half8{};
    }
  }

  float m_run[NRT], n_part[NRT];
  floatx4 acc[DT][NRT];
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    m_run[t] = kNegBig;
    n_part[t] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  for (int ci = 0; ci < sg.n_chunks; ++ci) {
    const int slot = P.seg_slots[sg.slot_off + ci];
    const int len = P.slot_len[slot];
    const size_t base = (static_cast<size_t>(slot) * H + h) * static_cast<size_t>(C) * D;
    const _Float16* kb = kpool + base;
    const _Float16* vb = vpool + base;
    for (int t0 = 0; t0 < len; t0 += 64) {
      const int nt = min(64, len - t0);
      // stage V rows of this block in LDS (zeros past the valid rows)
      constexpr int PIECES = 64 * D / 8;
#pragma unroll
      for (int pc = tid; pc < PIECES; pc += 256) {
        const int tok = pc / (D / 8), col = (pc % (D / 8)) * 8;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (tok < nt) val = *reinterpret_cast<const uint4*>(vb + static_cast<size_t>(t0 + tok) * D + col);
        uint32_t* dst = reinterpret_cast<uint32_t*>(v_lds + tok * VS + col);
        dst[0] = val.x;
        dst[1] = val.y;
        dst[2] = val.z;
        dst[3] = val.w;
      }
      // S^T = K Q^T for this wavefront's 16 tokens
      const int ktok = 16 * w + l16;
      half8 kf[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (ktok < nt)
          kf[s] = *reinterpret_cast<const half8*>(kb + static_cast<size_t>(t0 + ktok) * D + 32 * s + 8 * g);
        else
          kf[s] = half8{};
      }
      floatx4 sacc[NRT];
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        sacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (t < nrt) {
#pragma unroll
          for (int s = 0; s < KS; ++s)
            sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kf[s], qf[t][s], sacc[t], 0, 0, 0);
        }
      }
      // lane holds S^T[token 16w+4g+i][row 16t+l16]; scale, mask, row max
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        float lmax = kNegBig;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * w + 4 * g + i;
          const float x = tok < nt ? sacc[t][i] * P.qscale : -INFINITY;
          sacc[t][i] = x;
          lmax = fmaxf(lmax, x);
        }
        lmax = fmaxf(lmax, __shfl_xor(lmax, 16));
        lmax = fmaxf(lmax, __shfl_xor(lmax, 32));
        if (g == 0) red[w][16 * t + l16] = lmax;
      }
      __syncthreads();
      float alpha[NRT];
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        const int r = 16 * t + l16;
        const float bmax = fmaxf(fmaxf(red[0][r], red[1][r]), fmaxf(red[2][r], red[3][r]));
        const float mn = fmaxf(m_run[t], bmax);
        alpha[t] = fast_exp2(m_run[t] - mn);
        m_run[t] = mn;
        half4 ph;
        float ps = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ph[i] = static_cast<_Float16>(fast_exp2(sacc[t][i] - mn));
          ps += static_cast<float>(ph[i]);
        }
        n_part[t] = n_part[t] * alpha[t] + ps;
        *reinterpret_cast<half4*>(p_lds + r * PS + 16 * w + 4 * g) = ph;
      }
      __syncthreads();
      // O^T += V^T P^T over the block's 64 tokens (two k-steps of 32)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d0 = w * (D / 4) + 16 * dt;
#pragma unroll
        for (int t = 0; t < NRT; ++t) acc[dt][t] *= alpha[t];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          half8 va;
#pragma unroll
          for (int j = 0; j < 8; ++j) va[j] = v_lds[(32 * ks + 8 * g + j) * VS + d0 + l16];
#pragma unroll
          for (int t = 0; t < NRT; ++t) {
            if (t < nrt) {
              const half8 pb =
                  *reinterpret_cast<const half8*>(p_lds + (16 * t + l16) * PS + 32 * ks + 8 * g);
              acc[dt][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb, acc[dt][t], 0, 0, 0);
            }
          }
        }
      }
      __syncthreads();
    }
  }

  // row sums: combine lane groups and wavefronts
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    float ns = n_part[t];
    ns += __shfl_xor(ns, 16);
    ns += __shfl_xor(ns, 32);
    if (g == 0) red[w][16 * t + l16] = ns;
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    const int r = 16 * t + l16;
    if (r < nrows) {
      const size_t p = static_cast<size_t>(sg.part_base + (rb - sg.row_begin) + r);
      float* po = P.ws_o + (p * H + h) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<floatx4*>(po + w * (D / 4) + 16 * dt + 4 * g) = acc[dt][t];
      if (w == 0 && g == 0)
        P.ws_ml[p * H + h] = make_float2(m_run[t], red[0][r] + red[1][r] + red[2][r] + red[3][r]);
    }
  }
}

// fp32 chunk-first: the same schedule on the 16x16x4 fp32 matrix-core op.
// Operands are single floats (A: row l16, k = g; B: column l16, k = g).
template <int D, int NRT>
__global__ __launch_bounds__(256) void kcf_f32_kernel(KcfParams P) {
  constexpr int DT = D / 64;
  constexpr int VS = D + 1;
  constexpr int PS = 64 + 1;
  constexpr int R = 16 * NRT;
  __shared__ float v_lds[64 * VS];
  __shared__ float p_lds[R * PS];
  __shared__ float red[4][R];

  const CfSeg sg = P.segs[blockIdx.x];
  const int h = blockIdx.y, H = P.H, C = P.C;
  const int rb = sg.row_begin + static_cast<int>(blockIdx.z) * R;
  const int nrows = min(R, sg.row_end - rb);
  if (nrows <= 0) return;
  const int nrt = (nrows + 15) / 16;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const float* q = static_cast<const float*>(P.q);
  const float* kpool = static_cast<const float*>(P.kpool);
  const float* vpool = static_cast<const float*>(P.vpool);

  float m_run[NRT], n_part[NRT];
  floatx4 acc[DT][NRT];
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    m_run[t] = kNegBig;
    n_part[t] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt][t] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  for (int ci = 0; ci < sg.n_chunks; ++ci) {
    const int slot = P.seg_slots[sg.slot_off + ci];
    const int len = P.slot_len[slot];
    const size_t base = (static_cast<size_t>(slot) * H + h) * static_cast<size_t>(C) * D;
    const float* kb = kpool + base;
    const float* vb = vpool + base;
    for (int t0 = 0; t0 < len; t0 += 64) {
      const int nt = min(64, len - t0);
      constexpr int PIECES = 64 * D / 4;
      for (int pc = tid; pc < PIECES; pc += 256) {
        const int tok = pc / (D / 4), col = (pc % (D / 4)) * 4;
        float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
        if (tok < nt) val = *reinterpret_cast<const float4*>(vb + static_cast<size_t>(t0 + tok) * D + col);
        float* dst = v_lds + tok * VS + col;
        dst[0] = val.x;
        dst[1] = val.y;
        dst[2] = val.z;
        dst[3] = val.w;
      }
      const int ktok = 16 * w + l16;
      floatx4 sacc[NRT];
#pragma unroll
      for (int t = 0; t < NRT; ++t) sacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < D / 4; ++s) {
        const float a = ktok < nt ? kb[static_cast<size_t>(t0 + ktok) * D + 4 * s + g] : 0.f;
#pragma unroll
        for (int t = 0; t < NRT; ++t) {
          if (t < nrt) {
            const int r = 16 * t + l16;
            const float b = r < nrows ? q[(static_cast<size_t>(rb + r) * H + h) * D + 4 * s + g] : 0.f;
            sacc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, sacc[t], 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        float lmax = kNegBig;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tok = 16 * w + 4 * g + i;
          const float x = tok < nt ? sacc[t][i] * P.qscale : -INFINITY;
          sacc[t][i] = x;
          lmax = fmaxf(lmax, x);
        }
        lmax = fmaxf(lmax, __shfl_xor(lmax, 16));
        lmax = fmaxf(lmax, __shfl_xor(lmax, 32));
        if (g == 0) red[w][16 * t + l16] = lmax;
      }
      __syncthreads();
      float alpha[NRT];
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        const int r = 16 * t + l16;
        const float bmax = fmaxf(fmaxf(red[0][r], red[1][r]), fmaxf(red[2][r], red[3][r]));
        const float mn = fmaxf(m_run[t], bmax);
        alpha[t] = fast_exp2(m_run[t] - mn);
        m_run[t] = mn;
        float ps = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = fast_exp2(sacc[t][i] - mn);
          ps += p;
          p_lds[r * PS + 16 * w + 4 * g + i] = p;
        }
        n_part[t] = n_part[t] * alpha[t] + ps;
      }
      __syncthreads();
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d0 = w * (D / 4) + 16 * dt;
#pragma unroll
        for (int t = 0; t < NRT; ++t) acc[dt][t] *= alpha[t];
        for (int ks = 0; ks < 16; ++ks) {
          const float va = v_lds[(4 * ks + g) * VS + d0 + l16];
#pragma unroll
          for (int t = 0; t < NRT; ++t) {
            if (t < nrt) {
              const float pb = p_lds[(16 * t + l16) * PS + 4 * ks + g];
              acc[dt][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(va, pb, acc[dt][t], 0, 0, 0);
            }
          }
        }
      }
      __syncthreads();
    }
  }

#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    float ns = n_part[t];
    ns += __shfl_xor(ns, 16);
    ns += __shfl_xor(ns, 32);
    if (g == 0) red[w][16 * t + l16] = ns;
  }
  __syncthreads();
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    const int r = 16 * t + l16;
    if (r < nrows) {
      const size_t p = static_cast<size_t>(sg.part_base + (rb - sg.row_begin) + r);
      float* po = P.ws_o + (p * H + h) * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<floatx4*>(po + w * (D / 4) + 16 * dt + 4 * g) = acc[dt][t];
      if (w == 0 && g == 0)
        P.ws_ml[p * H + h] = make_float2(m_run[t], red[0][r] + red[1][r] + red[2][r] + red[3][r]);
    }
  }
}

// ---------------------------------------------------------------------------
// K/V copies for tree operations.

struct KvJobBatch {
  int32_t n;
  KvJob job[kKvJobsPerLaunch];
};

__global__ __launch_bounds__(256) void kkv_kernel(KvJobBatch b, const char* k, const char* v,
                                                  char* kpool, char* vpool, int32_t* slot_len,
                                                  int H, int row_bytes, int C) {
  const KvJob j = b.job[blockIdx.x];
  const int h = blockIdx.y;
  if (j.kind != 2) {
    const int units = row_bytes / 16;
    const size_t dst = ((static_cast<size_t>(j.dst_slot) * H + h) * C + j.dst_pos) *
                       static_cast<size_t>(row_bytes);
    const char *sk, *sv;
    size_t src, stride;
    if (j.kind == 0) {
      sk = k;
      sv = v;
      src = (static_cast<size_t>(j.src) * H + h) * static_cast<size_t>(row_bytes);
      stride = static_cast<size_t>(H) * row_bytes;
    } else {
      sk = kpool;
      sv = vpool;
      src = ((static_cast<size_t>(j.src) * H + h) * C + j.src_pos) * static_cast<size_t>(row_bytes);
      stride = row_bytes;
    }
    for (int i = threadIdx.x; i < j.n * units; i += blockDim.x) {
      const int r = i / units, u = i % units;
      const size_t so = src + r * stride + u * 16;
      const size_t dof = dst + static_cast<size_t>(r) * row_bytes + u * 16;
      *reinterpret_cast<uint4*>(kpool + dof) = *reinterpret_cast<const uint4*>(sk + so);
      *reinterpret_cast<uint4*>(vpool + dof) = *reinterpret_cast<const uint4*>(sv + so);
    }
  }
  if (h == 0 && threadIdx.x == 0) slot_len[j.dst_slot] = j.kind == 2 ? j.dst_pos : j.dst_pos + j.n;
}

template <typename T, int D>
void launch_kcf_t(const AttnArgs& a, const DevWork& w, hipStream_t s) {
  KcfParams P{a.q, a.kpool, a.vpool, a.slot_len, w.segs, w.seg_slots, a.ws_o,
              reinterpret_cast<float2*>(a.ws_ml), a.H, a.C, a.qscale};
  const int rows = w.max_seg_rows;
  const int nrt = rows <= 16 ? 1 : rows <= 32 ? 2 : 4;
  const int zb = (rows + 16 * nrt - 1) / (16 * nrt);
  const dim3 grid(w.n_segs, a.H, zb);
  if constexpr (sizeof(T) == 2) {
    if (nrt == 1) kcf_f16_kernel<D, 1><<<grid, 256, 0, s>>>(P);
    else if (nrt == 2) kcf_f16_kernel<D, 2><<<grid, 256, 0, s>>>(P);
    else kcf_f16_kernel<D, 4><<<grid, 256, 0, s>>>(P);
  } else {
    if (nrt == 1) kcf_f32_kernel<D, 1><<<grid, 256, 0, s>>>(P);
    else if (nrt == 2) kcf_f32_kernel<D, 2><<<grid, 256, 0, s>>>(P);
    else kcf_f32_kernel<D, 4><<<grid, 256, 0, s>>>(P);
  }
}

template <typename T, int D>
hipError_t launch_all(const AttnArgs& a, const DevWork& w, hipStream_t s, int mask) {
  if ((mask & 1) && w.n_segs > 0) launch_kcf_t<T, D>(a, w, s);
  if ((mask & 2) && w.n_items > 0) {
    KsfParams P{a.q, a.o, a.kpool, a.vpool, a.slot_len, w.items, w.priv_slot, w.part_ptr, w.parts,
                a.ws_o, reinterpret_cast<float2*>(a.ws_ml), a.H, a.C, a.qscale};
    ksf_kernel<T, D><<<dim3(w.n_items, a.H), 256, 0, s>>>(P);
  }
  if ((mask & 4) && w.n_mg > 0) {
    KmgParams P{a.o, w.mg_rows, w.part_ptr, w.parts, a.ws_o, reinterpret_cast<const float2*>(a.ws_ml),
                a.H};
    kmg_kernel<T, D><<<dim3(w.n_mg, a.H), 64, 0, s>>>(P);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, const DevWork& w, hipStream_t s, int mask) {
  if (a.dtype == 0) {
    if (a.D == 128) return launch_all<_Float16, 128>(a, w, s, mask);
    if (a.D == 64) return launch_all<_Float16, 64>(a, w, s, mask);
  } else {
    if (a.D == 128) return launch_all<float, 128>(a, w, s, mask);
    if (a.D == 64) return launch_all<float, 64>(a, w, s, mask);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_kv_jobs(const KvJob* jobs, int n, int dtype, int H, int D, int C, const void* k,
                          const void* v, void* kpool, void* vpool, int32_t* slot_len,
                          hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (n > kKvJobsPerLaunch) return hipErrorInvalidValue;
  KvJobBatch b;
  b.n = n;
  for (int i = 0; i < n; ++i) b.job[i] = jobs[i];
  const int row_bytes = D * (dtype == 0 ? 2 : 4);
  kkv_kernel<<<dim3(n, H), 256, 0, stream>>>(b, static_cast<const char*>(k),
                                             static_cast<const char*>(v), static_cast<char*>(kpool),
                                             static_cast<char*>(vpool), slot_len, H, row_bytes, C);
  return hipGetLastError();
}

}  // namespace ca
