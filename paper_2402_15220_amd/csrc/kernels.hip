// gfx950 (MI355X) kernels for decode attention over a prefix-tree, chunked
// KV cache with the two-phase partition of ChunkAttention (arXiv 2402.15220,
// Section 3.2).
//
// Pools: K and V, each [slot][head][c][d]; slot_len[slot] holds the number of
// valid rows of every slot. q and o: [B][H][d] in tree row order.
// Softmax runs in base 2: scores are multiplied by scale*log2(e), so partial
// maxima stored in the workspace are in log2 units.
//
// Two schedules: the phases as consecutive launches, or both in ONE launch
// (tpp_kernel) whose first blocks are chunk-first items and the rest
// sequence-first items, so the latency-bound chunk-first work overlaps the
// bandwidth-bound stream.
//   kcf  chunk-first phase (Algorithm 1, Eqn 1). One workgroup per (segment
//        of shared chunks, head, block of <= 16*NRT covered rows). For every
//        64-token block of a chunk it forms S^T = K Q^T on the matrix cores
//        (the covered query rows batched as the N dimension), updates the
//        online softmax per row, and accumulates O^T = V^T P^T, again on the
//        matrix cores. It writes one unnormalised partial (O, m, n) per row.
//   ksf  sequence-first phase (Algorithm 2). One workgroup per (row, head,
//        piece of the row's private chunks): a bandwidth-bound pass with
//        16-byte loads, sub-wavefront DPP reductions for q.k and per-lane
//        online softmax. An item that owns its row folds the row's
//        chunk-first partials (sequential schedule) and writes O/n; otherwise
//        it writes a partial.
//   kmg  merge epilogue (Algorithm 2's attn_reduce over the partials, Eqn 2,
//        then O/n) for every row that has partials.
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

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ float readlane_f(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}

// attn_reduce (Eqn 2) of partials parts[k0..k1) into (m, n, acc), a whole
// wavefront cooperating: the lanes read up to 64 partial maxima at once, the
// common maximum rescales everything once, then every lane accumulates its
// d-slice [d0, d0+E) of each partial's O (independent loads, in flight
// together). Call with all 64 lanes active.
template <int E>
__device__ __forceinline__ void fold_parts(int k0, int k1, const int32_t* parts, const float* ws_o,
                                           const float2* ws_ml, int H, int D, int h, int d0,
                                           int lane, float& m, float& n, float* acc) {
  for (int b0 = k0; b0 < k1; b0 += 64) {
    const int nb = min(64, k1 - b0);
    int pidx = 0;
    float pm = kNegBig, pn = 0.f;
    if (lane < nb) {
      pidx = parts[b0 + lane];
      const float2 ml = ws_ml[static_cast<size_t>(pidx) * H + h];
      pm = ml.x;
      pn = ml.y;
    }
    const float M = fmaxf(m, wave_max(pm));
    const float wself = fast_exp2(m - M);
    const float wp = lane < nb ? fast_exp2(pm - M) : 0.f;
    n = n * wself + wave_sum(wp * pn);
#pragma unroll
    for (int j = 0; j < E; ++j) acc[j] *= wself;
#pragma unroll 4
    for (int k = 0; k < nb; ++k) {
      const int pk = __builtin_amdgcn_readlane(pidx, k);
      const float wk = readlane_f(wp, k);
      const float* po = ws_o + (static_cast<size_t>(pk) * H + h) * D + d0;
#pragma unroll
      for (int j = 0; j < E; j += 4) {
        const float4 x = *reinterpret_cast<const float4*>(po + j);
        acc[j] = fmaf(wk, x.x, acc[j]);
        acc[j + 1] = fmaf(wk, x.y, acc[j + 1]);
        acc[j + 2] = fmaf(wk, x.z, acc[j + 2]);
        acc[j + 3] = fmaf(wk, x.w, acc[j + 3]);
      }
    }
    m = M;
  }
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
constexpr int ksf_lds_bytes() {
  return 4 * (D * sizeof(T) / 16) * (16 / static_cast<int>(sizeof(T)) + 2) * 4;
}

template <typename T, int D>
__device__ __forceinline__ void ksf_block(const KsfParams& P, int item, int h, char* lds) {
  using E = Elem<T>;
  constexpr int EPL = E::kPerVec;
  constexpr int LPT = D / EPL;
  constexpr int TPW = 64 / LPT;
  constexpr int TPS = TPW * 4;
  constexpr int U = 64 / TPS;
  static_assert(U >= 1 && TPS * U == 64, "step must cover 64 tokens");

  const SfItem it = P.items[item];
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

  const T* kpool = static_cast<const T*>(P.kpool) + static_cast<size_t>(h) * C * D + sub * EPL;
  const T* vpool = static_cast<const T*>(P.vpool) + static_cast<size_t>(h) * C * D + sub * EPL;
  const size_t slot_stride = static_cast<size_t>(H) * C * D;
  const int tok_off = w * TPW + tr;  // this lane's token within a step (u = 0)

  auto load_step = [&](uint4* kr, uint4* vr, int slot, int t0, int len) {
    const T* kb = kpool + slot * slot_stride;
    const T* vb = vpool + slot * slot_stride;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tok = t0 + u * TPS + tok_off;
      if (tok < len) {
        kr[u] = *reinterpret_cast<const uint4*>(kb + static_cast<size_t>(tok) * D);
        vr[u] = *reinterpret_cast<const uint4*>(vb + static_cast<size_t>(tok) * D);
      } else {
        kr[u] = make_uint4(0, 0, 0, 0);
        vr[u] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  // online softmax over one 64-token step (Eqn 1 for the step, folded by Eqn 2)
  auto do_step = [&](const uint4* kr, const uint4* vr, int t0, int len) {
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
      const int tok = t0 + u * TPS + tok_off;
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
  };

  // Chunks are taken 64 at a time: lane i holds the slot and length of chunk
  // i of the group, broadcast with readlane. The next step's K/V loads are
  // issued before the current step is computed.
  for (int g0 = it.cb; g0 < it.ce; g0 += 64) {
    const int gn = min(64, it.ce - g0);
    int my_slot = 0, my_len = 0;
    if (lane < gn) {
      my_slot = P.priv_slot[g0 + lane];
      my_len = P.slot_len[my_slot];
    }
    int j = 0, t0 = 0;
    int slot = __builtin_amdgcn_readlane(my_slot, 0);
    int len = __builtin_amdgcn_readlane(my_len, 0);
    uint4 kr[U], vr[U];
    load_step(kr, vr, slot, t0, len);
    while (true) {
      int j2 = j, t02 = t0 + 64, slot2 = slot, len2 = len;
      if (t02 >= len) {
        j2 = j + 1;
        t02 = 0;
        if (j2 < gn) {
          slot2 = __builtin_amdgcn_readlane(my_slot, j2);
          len2 = __builtin_amdgcn_readlane(my_len, j2);
        }
      }
      const bool more = j2 < gn;
      uint4 kn[U], vn[U];
      if (more) load_step(kn, vn, slot2, t02, len2);
      do_step(kr, vr, t0, len);
      if (!more) break;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        kr[u] = kn[u];
        vr[u] = vn[u];
      }
      j = j2;
      t0 = t02;
      slot = slot2;
      len = len2;
    }
  }

  // combine the token-row groups of this wavefront (every lane of a d-slice
  // ends with the same state)
#pragma unroll
  for (int off = LPT; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m, off);
    const float no = __shfl_xor(n, off);
    float ao[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) ao[j] = __shfl_xor(acc[j], off);
    fold<EPL>(m, n, acc, mo, no, ao);
  }
  // combine the four wavefronts in wavefront 0
  auto st = reinterpret_cast<float (*)[LPT][EPL + 2]>(lds);
  if (tr == 0) {
    st[w][sub][0] = m;
    st[w][sub][1] = n;
#pragma unroll
    for (int j = 0; j < EPL; ++j) st[w][sub][2 + j] = acc[j];
  }
  __syncthreads();
  if (w != 0) return;
#pragma unroll
  for (int ww = 1; ww < 4; ++ww) fold<EPL>(m, n, acc, st[ww][sub][0], st[ww][sub][1], &st[ww][sub][2]);

  if (it.out_part < 0) {
    // fold the row's chunk-first partials (Algorithm 2), then O/n
    fold_parts<EPL>(P.part_ptr[it.row], P.part_ptr[it.row + 1], P.parts, P.ws_o, P.ws_ml, H, D,
                    h, sub * EPL, lane, m, n, acc);
    if (tr != 0) return;
    const float inv = 1.f / n;
#pragma unroll
    for (int j = 0; j < EPL; ++j) acc[j] *= inv;
    *reinterpret_cast<uint4*>(static_cast<T*>(P.o) + (static_cast<size_t>(it.row) * H + h) * D +
                              sub * EPL) = E::pack(acc);
  } else {
    if (tr != 0) return;
    float* po = P.ws_o + (static_cast<size_t>(it.out_part) * H + h) * D + sub * EPL;
#pragma unroll
    for (int j = 0; j < EPL; j += 4)
      *reinterpret_cast<float4*>(po + j) = make_float4(acc[j], acc[j + 1], acc[j + 2], acc[j + 3]);
    if (sub == 0) P.ws_ml[static_cast<size_t>(it.out_part) * H + h] = make_float2(m, n);
  }
}

// ---------------------------------------------------------------------------
// Merge epilogue: rows whose result is spread over several partials.

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
  const int row = P.mg_rows[blockIdx.x];
  const int h = blockIdx.y, H = P.H;
  const int lane = threadIdx.x;
  // lanes 0..D/4-1 own four consecutive d each; the rest mirror lane % (D/4)
  const int d0 = (lane % (D / 4)) * 4;
  float m = kNegBig, n = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
  fold_parts<4>(P.part_ptr[row], P.part_ptr[row + 1], P.parts, P.ws_o, P.ws_ml, H, D, h, d0, lane,
                m, n, acc);
  if (lane >= D / 4) return;
  const float inv = 1.f / n;
  T* o = static_cast<T*>(P.o) + (static_cast<size_t>(row) * H + h) * D + d0;
#pragma unroll
  for (int j = 0; j < 4; ++j) o[j] = static_cast<T>(acc[j] * inv);
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
constexpr int kcf_f16_lds_bytes() {
  return 64 * (D + 2) * 2 + 16 * NRT * (64 + 8) * 2 + 4 * 16 * NRT * 4;
}

template <int D, int NRT>
__device__ __forceinline__ void kcf_f16_block(const KcfParams& P, int seg, int z, int h, char* lds) {
  constexpr int KS = D / 32;  // 16x16x32 steps over d for S^T
  constexpr int DT = D / 64;  // 16-wide d tiles per wavefront for O^T
  constexpr int VS = D + 2;   // V row stride in LDS (halves)
  constexpr int PS = 64 + 8;  // P row stride in LDS (halves), keeps 16-byte row alignment
  constexpr int R = 16 * NRT;
  _Float16* v_lds = reinterpret_cast<_Float16*>(lds);
  _Float16* p_lds = v_lds + 64 * VS;
  auto red = reinterpret_cast<float (*)[R]>(p_lds + R * PS);

  const CfSeg sg = P.segs[seg];
  const int H = P.H, C = P.C;
  const int rb = sg.row_begin + z * R;
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
constexpr int kcf_f32_lds_bytes() {
  return 64 * (D + 1) * 4 + 16 * NRT * (64 + 1) * 4 + 4 * 16 * NRT * 4;
}

template <int D, int NRT>
__device__ __forceinline__ void kcf_f32_block(const KcfParams& P, int seg, int z, int h, char* lds) {
  constexpr int DT = D / 64;
  constexpr int VS = D + 1;
  constexpr int PS = 64 + 1;
  constexpr int R = 16 * NRT;
  float* v_lds = reinterpret_cast<float*>(lds);
  float* p_lds = v_lds + 64 * VS;
  auto red = reinterpret_cast<float (*)[R]>(p_lds + R * PS);

  const CfSeg sg = P.segs[seg];
  const int H = P.H, C = P.C;
  const int rb = sg.row_begin + z * R;
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

// Fused schedule, one launch for both phases: blocks [0, n_cf) run
// chunk-first work items (dispatched first), the remaining blocks run
// sequence-first items; both write partial results and the merge epilogue
// combines them. Sequential schedule: chunk-first launch, then a
// sequence-first launch whose items fold the finished chunk-first partials
// themselves (the merge epilogue only finishes split rows).
struct TppParams {
  KcfParams cf;
  KsfParams sf;
  int n_cf;        // chunk-first blocks: n_segs * zb * H
  int zb;          // row blocks per segment
  int block_base;  // first block index of this launch
};

template <typename T, int D, int NRT>
constexpr int tpp_lds_bytes() {
  constexpr int cf = sizeof(T) == 2 ? kcf_f16_lds_bytes<D, NRT>() : kcf_f32_lds_bytes<D, NRT>();
  constexpr int sf = ksf_lds_bytes<T, D>();
  return cf > sf ? cf : sf;
}

template <typename T, int D, int NRT>
__global__ __launch_bounds__(256, 4) void tpp_kernel(TppParams P) {
  __shared__ __attribute__((aligned(16))) char lds[tpp_lds_bytes<T, D, NRT>()];
  const int b = static_cast<int>(blockIdx.x) + P.block_base;
  const int H = P.sf.H;
  if (b < P.n_cf) {
    const int h = b % H;
    const int rest = b / H;
    const int z = rest % P.zb;
    const int seg = rest / P.zb;
    if constexpr (sizeof(T) == 2)
      kcf_f16_block<D, NRT>(P.cf, seg, z, h, lds);
    else
      kcf_f32_block<D, NRT>(P.cf, seg, z, h, lds);
  } else {
    const int bb = b - P.n_cf;
    ksf_block<T, D>(P.sf, bb / H, bb % H, lds);
  }
}

// The phases as separate launches (same block functions, own resources).
template <typename T, int D, int NRT>
__global__ __launch_bounds__(256) void kcf_kernel(KcfParams P, int zb) {
  constexpr int L = sizeof(T) == 2 ? kcf_f16_lds_bytes<D, NRT>() : kcf_f32_lds_bytes<D, NRT>();
  __shared__ __attribute__((aligned(16))) char lds[L];
  const int b = static_cast<int>(blockIdx.x);
  const int h = b % P.H;
  const int rest = b / P.H;
  if constexpr (sizeof(T) == 2)
    kcf_f16_block<D, NRT>(P, rest / zb, rest % zb, h, lds);
  else
    kcf_f32_block<D, NRT>(P, rest / zb, rest % zb, h, lds);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void ksf_kernel(KsfParams P) {
  __shared__ __attribute__((aligned(16))) char lds[ksf_lds_bytes<T, D>()];
  const int b = static_cast<int>(blockIdx.x);
  ksf_block<T, D>(P, b / P.H, b % P.H, lds);
}

template <typename T, int D, int NRT>
void launch_phases(const TppParams& P, int n_sf, bool fused, int mask, hipStream_t s) {
  if (fused && (mask & 1) && (mask & 2)) {
    const int grid = P.n_cf + n_sf;
    if (grid > 0) tpp_kernel<T, D, NRT><<<grid, 256, 0, s>>>(P);
    return;
  }
  if ((mask & 1) && P.n_cf > 0) kcf_kernel<T, D, NRT><<<P.n_cf, 256, 0, s>>>(P.cf, P.zb);
  if ((mask & 2) && n_sf > 0) ksf_kernel<T, D><<<n_sf, 256, 0, s>>>(P.sf);
}

template <typename T, int D>
hipError_t launch_all(const AttnArgs& a, const DevWork& w, hipStream_t s, int mask) {
  TppParams P;
  P.cf = KcfParams{a.q, a.kpool, a.vpool, a.slot_len, w.segs, w.seg_slots, a.ws_o,
                   reinterpret_cast<float2*>(a.ws_ml), a.H, a.C, a.qscale};
  P.sf = KsfParams{a.q, a.o, a.kpool, a.vpool, a.slot_len, w.items, w.priv_slot, w.part_ptr,
                   w.parts, a.ws_o, reinterpret_cast<float2*>(a.ws_ml), a.H, a.C, a.qscale};
  const int rows = w.max_seg_rows;
  const int nrt = rows <= 16 ? 1 : rows <= 32 ? 2 : 4;
  P.zb = rows > 0 ? (rows + 16 * nrt - 1) / (16 * nrt) : 1;
  P.n_cf = w.n_segs * P.zb * a.H;
  P.block_base = 0;
  const int n_sf = w.n_items * a.H;
  if (nrt == 1) launch_phases<T, D, 1>(P, n_sf, w.fused, mask, s);
  else if (nrt == 2) launch_phases<T, D, 2>(P, n_sf, w.fused, mask, s);
  else launch_phases<T, D, 4>(P, n_sf, w.fused, mask, s);
  if ((mask & 4) && w.n_mg > 0) {
    KmgParams M{a.o, w.mg_rows, w.part_ptr, w.parts, a.ws_o, reinterpret_cast<const float2*>(a.ws_ml),
                a.H};
    kmg_kernel<T, D><<<dim3(w.n_mg, a.H), 64, 0, s>>>(M);
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
