// gfx950 (MI355X) kernels for decode attention over a prefix-tree, chunked
// KV cache with the two-phase partition of ChunkAttention (arXiv 2402.15220,
// Section 3.2).
//
// Pools: K and V tiles of c x d elements per (slot, head) at slot and head
// strides; slot_len[slot] holds the number of valid rows of every slot.
// q and o: [B][H][d], in tree row order or, through a row map, in the
// caller's order. Softmax runs in base 2: scores are multiplied by
// scale*log2(e), so partial maxima stored in the workspace are in log2 units.
//
// Schedules (ca_set_tuning): the phases as consecutive launches (0); both in
// ONE launch (tpp_kernel) whose first blocks are chunk-first items and the
// rest sequence-first items, so the latency-bound chunk-first work overlaps
// the bandwidth-bound stream, with a merge launch (1) or with the last
// contributor of each row merging inside the launch (2, default); the phases
// on two streams (3); and the partial-free serial reduction (4), one
// chunk-first launch per position along the rows' paths.
//   kcf  chunk-first phase (Algorithm 1, Eqn 1). One workgroup per (segment
//        of shared chunks, head, block of <= 16*NRT covered rows). For every
//        64-token block of a chunk it forms S^T = K Q^T on the matrix cores
//        (the covered query rows batched as the N dimension), updates the
//        online softmax per row, and accumulates O^T = V^T P^T, again on the
//        matrix cores. It writes one unnormalised partial (O, m, n) per row
//        (or, in schedule 4, folds it into the row's accumulator).
//   ksf  sequence-first phase (Algorithm 2). One workgroup per (row, head,
//        piece of the row's private chunks): a bandwidth-bound pass with
//        16-byte loads, sub-wavefront DPP reductions for q.k and per-lane
//        online softmax. An item that owns its row folds the row's
//        chunk-first partials and writes O/n; otherwise it writes a partial.
//   kmg  merge epilogue (Algorithm 2's attn_reduce over the partials, Eqn 2,
//        then O/n) for every row that has partials.
//   kkv  K/V row copies for tree operations (new chunks, split tails).
// The prefill kernel lives in prefill.hip.
#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

#include "device_common.hpp"
#include "kernels.hpp"

namespace ca {
namespace {

// Row of q and o that holds tree row `row`: the caller's order when a row
// map is given, else tree order.
__device__ __forceinline__ int io_row(const int32_t* row_map, int row) {
  return row_map ? row_map[row] : row;
}

// Byte offset of element d of partial p, head h in the partial-O workspace.
__device__ __forceinline__ uint32_t part_off(int p, int H, int D, int h, int d) {
  return ((static_cast<uint32_t>(p) * H + h) * D + d) * 4u;
}

// attn_reduce (Eqn 2) of partials parts[k0..k1) into (m, n, acc), a whole
// wavefront cooperating. The lanes read up to 64 partial maxima at once and
// one common maximum rescales everything once. The wavefront is G groups of
// 64/G lanes; each lane owns the d-slice [d0, d0+E) and its group takes
// every G-th partial, all loads of a batch (NB partials per group) issued
// before the first is used; the group sums are added at the end, so every
// lane returns the whole result for its slice. (m, n, acc) must be the same
// in every group on entry. A skipped partial (`skip`, this block's own) or
// an absent one gets weight 0 and reads a valid partial in its place, never
// unwritten workspace. DEV selects device-scope loads (partials written by
// other blocks of the same launch). Call with all 64 lanes active.
template <int E, int G, bool DEV>
__device__ __forceinline__ void fold_parts(int k0, int k1, const int32_t* parts, const float* ws_o,
                                           uint32_t o_bytes, const float2* ws_ml, int H, int D,
                                           int h, int d0, int lane, float& m, float& n, float* acc,
                                           int skip = -1) {
  constexpr int NB = 32 / E;
  static_assert(E % 4 == 0 && NB >= 1 && G >= 1 && 64 % G == 0, "fold layout");
  const int gi = lane / (64 / G);
  const __amdgpu_buffer_rsrc_t rs = part_rsrc(ws_o, o_bytes);
  if (gi != 0) {
#pragma unroll
    for (int j = 0; j < E; ++j) acc[j] = 0.f;
  }
  for (int b0 = k0; b0 < k1; b0 += 64) {
    const int nb = min(64, k1 - b0);
    int pidx = lane < nb ? parts[b0 + lane] : -1;
    const bool valid = pidx >= 0 && pidx != skip;
    float pm = kNegBig, pn = 0.f;
    if (valid) {
      const float* ml = reinterpret_cast<const float*>(ws_ml + static_cast<size_t>(pidx) * H + h);
      if constexpr (DEV) {
        pm = ld_dev(ml);
        pn = ld_dev(ml + 1);
      } else {
        pm = ml[0];
        pn = ml[1];
      }
    }
    const unsigned long long vm = __ballot(valid);
    if (vm == 0) continue;  // uniform
    if (!valid) pidx = __builtin_amdgcn_readlane(pidx, __builtin_ctzll(vm));
    const float M = fmaxf(m, wave_max(pm));
    const float wself = fast_exp2(m - M);
    const float wp = valid ? fast_exp2(pm - M) : 0.f;
    n = n * wself + wave_sum(wp * pn);
#pragma unroll
    for (int j = 0; j < E; ++j) acc[j] *= wself;
    const int kend = 64 - __builtin_clzll(vm);  // one past the last valid lane
    for (int kb = 0; kb < kend; kb += NB * G) {
      float x[NB][E];
      float wk[NB];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int k = kb + G * u + gi;
        const int kc = min(k, 63);
        const int pk = __shfl(pidx, kc);
        wk[u] = k < 64 ? __shfl(wp, kc) : 0.f;
#pragma unroll
        for (int j = 0; j < E; j += 4) {
          float4 v;
          if constexpr (DEV) {
            v = ld_dev4(rs, part_off(pk, H, D, h, d0 + j));
          } else {
            v = *reinterpret_cast<const float4*>(ws_o + (static_cast<size_t>(pk) * H + h) * D + d0 + j);
          }
          x[u][j] = v.x;
          x[u][j + 1] = v.y;
          x[u][j + 2] = v.z;
          x[u][j + 3] = v.w;
        }
      }
#pragma unroll
      for (int u = 0; u < NB; ++u) {
#pragma unroll
        for (int j = 0; j < E; ++j) acc[j] = fmaf(wk[u], x[u][j], acc[j]);
      }
    }
    m = M;
  }
#pragma unroll
  for (int j = 0; j < E; ++j) {
#pragma unroll
    for (int off = 64 / G; off < 64; off <<= 1) acc[j] += __shfl_xor(acc[j], off);
  }
}

// fold_parts for at most 64 partials whose indices are already in lanes
// (lane k holds the k-th, pidx < 0 past the end): the maxima and every
// partial O vector are requested together, one round trip instead of a
// chain of index, maximum and vector loads, then folded (Eqn 2) with one
// common maximum. Same lane layout, arguments and result as fold_parts.
template <int E, int G, bool DEV>
__device__ __forceinline__ void fold_parts_lanes(int pidx, const float* ws_o, uint32_t o_bytes,
                                                 const float2* ws_ml, int H, int D, int h, int d0,
                                                 int lane, float& m, float& n, float* acc, int skip) {
  constexpr int NB = 32 / E;  // partials per group per pass
  static_assert(E % 4 == 0 && NB >= 1 && G >= 1 && 64 % G == 0, "fold layout");
  const int gi = lane / (64 / G);
  const bool valid = pidx >= 0 && pidx != skip;
  const unsigned long long vm = __ballot(valid);
  if (vm == 0) return;  // uniform: nothing to fold
  // an absent or skipped partial reads a valid one in its place (weight 0)
  const int ps = valid ? pidx : __builtin_amdgcn_readlane(pidx, __builtin_ctzll(vm));
  const __amdgpu_buffer_rsrc_t rs = part_rsrc(ws_o, o_bytes);
  float pm = kNegBig, pn = 0.f;
  if (valid) {
    const float* ml = reinterpret_cast<const float*>(ws_ml + static_cast<size_t>(ps) * H + h);
    if constexpr (DEV) {
      pm = ld_dev(ml);
      pn = ld_dev(ml + 1);
    } else {
      pm = ml[0];
      pn = ml[1];
    }
  }
  const int kend = 64 - __builtin_clzll(vm);  // one past the last valid lane
  auto load_pass = [&](int kb, float (*x)[E]) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int kc = min(kb + G * u + gi, 63);
      const int pk = __shfl(ps, kc);
#pragma unroll
      for (int j = 0; j < E; j += 4) {
        float4 v;
        if constexpr (DEV) {
          v = ld_dev4(rs, part_off(pk, H, D, h, d0 + j));
        } else {
          v = *reinterpret_cast<const float4*>(ws_o + (static_cast<size_t>(pk) * H + h) * D + d0 + j);
        }
        x[u][j] = v.x;
        x[u][j + 1] = v.y;
        x[u][j + 2] = v.z;
        x[u][j + 3] = v.w;
      }
    }
  };
  float x[NB][E];
  load_pass(0, x);  // in flight with the maxima
  const float M = fmaxf(m, wave_max(pm));
  const float wself = fast_exp2(m - M);
  const float wp = valid ? fast_exp2(pm - M) : 0.f;
  n = n * wself + wave_sum(wp * pn);
#pragma unroll
  for (int j = 0; j < E; ++j) acc[j] = gi == 0 ? acc[j] * wself : 0.f;
  for (int kb = 0; kb < kend; kb += NB * G) {
    if (kb > 0) load_pass(kb, x);
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int k = kb + G * u + gi;
      const float wk = k < 64 ? __shfl(wp, min(k, 63)) : 0.f;
#pragma unroll
      for (int j = 0; j < E; ++j) acc[j] = fmaf(wk, x[u][j], acc[j]);
    }
  }
  m = M;
#pragma unroll
  for (int j = 0; j < E; ++j) {
#pragma unroll
    for (int off = 64 / G; off < 64; off <<= 1) acc[j] += __shfl_xor(acc[j], off);
  }
}

// Finish row `row`, head h from its partials (Eqn 2, then O/n) and write o.
// One wavefront; lanes [0, D/4) own four consecutive d each. DEV selects
// device-scope loads (partials written by other blocks of the same launch).
template <typename T, int D, bool DEV>
__device__ __forceinline__ void finish_row(const int32_t* part_ptr, const int32_t* parts,
                                           const float* ws_o, uint32_t o_bytes, const float2* ws_ml,
                                           void* o, const int32_t* row_map, int H, int row,
                                           int h, int lane) {
  const int d0 = (lane % (D / 4)) * 4;
  float m = kNegBig, n = 0.f, acc[4] = {0.f, 0.f, 0.f, 0.f};
  fold_parts<4, 256 / D, DEV>(part_ptr[row], part_ptr[row + 1], parts, ws_o, o_bytes, ws_ml, H, D,
                              h, d0, lane, m, n, acc);
  if (lane < D / 4) {
    const float inv = 1.f / n;
    T* out = static_cast<T*>(o) + (static_cast<size_t>(io_row(row_map, row)) * H + h) * D + d0;
#pragma unroll
    for (int j = 0; j < 4; ++j) out[j] = static_cast<T>(acc[j] * inv);
  }
}


// ---------------------------------------------------------------------------
// Sequence-first phase.

struct KsfParams {
  const void* q;
  void* o;
  const void* kpool;
  const void* vpool;
  int64_t ss, hs;  // pool strides of a slot and of a head (elements)
  const int32_t* slot_len;
  const SfItem* items;
  const int32_t* priv_slot;
  const int32_t* part_ptr;
  const int32_t* parts;
  float* ws_o;
  float2* ws_ml;
  uint32_t o_bytes;  // bytes of the partial-O region at ws_o
  int H;
  int C;
  float qscale;
  int32_t* cnt;  // partial-writing schedules: per (row, head) arrival counters, else null
  const int32_t* row_map;  // tree row -> row of q and o (null: tree order)
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

  const int H = P.H, C = P.C;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int sub = lane % LPT, tr = lane / LPT;

  // Everything the stream needs first is requested in the first round trip
  // or right after it: the item record (uniform) and, from the record's
  // inline copy, the slots of the first kSfInline chunks (one per lane);
  // then the first step's K/V rows, the first chunk's length, q, the row's
  // partial indices and the other lanes' lengths. No load waits on a chain
  // of other loads before the stream starts.
  const SfItem* itp = P.items + item;
  const SfItem it = *itp;
  int slot_lo = lane < kSfInline ? itp->slot[lane] : 0;

  const T* kpool = static_cast<const T*>(P.kpool) + h * P.hs + sub * EPL;
  const T* vpool = static_cast<const T*>(P.vpool) + h * P.hs + sub * EPL;
  const size_t slot_stride = static_cast<size_t>(P.ss);
  const int tok_off = w * TPW + tr;  // this lane's token within a step (u = 0)

  // Loads are unconditional (no branches, so the compiler can count them):
  // rows past the chunk's length re-read its last row, a finite valid row;
  // their scores are masked to -inf, so they add exactly 0 * v = 0.
  // Private rows are read once per call: the V rows are loaded non-temporal
  // so that half of this stream does not displace the shared chunks, which
  // the chunk-first blocks read once per 16 covered rows (measured: 15-18%
  // faster with long shared runs and 6-7% faster with evicted caches; with
  // both K and V non-temporal, back-to-back calls on a working set just above
  // the 256 MB Infinity Cache lost its reuse and were 5% slower).
  auto load_step = [&](uint4* kr, uint4* vr, int slot, int t0, int len) {
    const T* kb = kpool + slot * slot_stride;
    const T* vb = vpool + slot * slot_stride;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int tok = t0 + u * TPS + tok_off;
      const size_t row = static_cast<size_t>(min(tok, len - 1)) * D;
      kr[u] = *reinterpret_cast<const uint4*>(kb + row);
      vr[u] = __builtin_bit_cast(
          uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vb + row)));
    }
  };

  const int n_chunks = it.ce - it.cb;
  const int cm = min(C, 64);  // rows of a chunk's first step when the chunk is full
  uint4 kr[U], vr[U];
  // The first step of the first chunk goes out before the chunk's length
  // is known, as if the chunk were full (rows clamped to the tile, so in
  // bounds); a shorter chunk is requested again with the right clamp below
  // (rows past its length may hold anything, even NaN, and are never used).
  if (n_chunks > 0) load_step(kr, vr, it.slot[0], 0, cm);
  const int gn0 = min(64, n_chunks);
  int slot_hi = 0;
  if (lane >= it.n_inline && lane < gn0) slot_hi = P.priv_slot[it.cb + lane];
  const uint4 qr = *reinterpret_cast<const uint4*>(static_cast<const T*>(P.q) +
                                                   (static_cast<size_t>(io_row(P.row_map, it.row)) * H + h) * D +
                                                   sub * EPL);
  const int np = it.part_e - it.part_b;
  int pidx = -1;
  if (w == 0 && lane < np && np <= 64) pidx = P.parts[it.part_b + lane];
  const int len0 = n_chunks > 0 ? P.slot_len[it.slot[0]] : 0;
  int len_lo = lane < it.n_inline ? P.slot_len[slot_lo] : 0;
  float qf[EPL];
  E::unpack(qr, qf);

  float m = kNegBig, n = 0.f, acc[EPL];
#pragma unroll
  for (int j = 0; j < EPL; ++j) acc[j] = 0.f;

  // online softmax over one 64-token step (Eqn 1 for the step, folded by Eqn 2)
  auto do_step = [&](const uint4* kr_, const uint4* vr_, int t0, int len) {
    float s[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[EPL];
      E::unpack(kr_[u], kf);
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
      E::unpack(vr_[u], vf);
#pragma unroll
      for (int j = 0; j < EPL; ++j) acc[j] = fmaf(p, vf[j], acc[j]);
    }
    m = mn;
  };

  if (n_chunks > 0) {
    // chunks are taken 64 at a time: lane i holds the slot and length of
    // chunk i of the group, broadcast with readlane; in the first group the
    // first kSfInline come from the record (slot_lo, len_lo) and the others
    // from priv_slot (slot_hi, len_hi), so the early chunks never wait for
    // the later ones' lengths
    if (len0 < cm) load_step(kr, vr, it.slot[0], 0, len0);  // uniform; rare
    do_step(kr, vr, 0, len0);
    int len_hi = 0;
    if (lane >= it.n_inline && lane < gn0) len_hi = P.slot_len[slot_hi];
    int jj = 0, t0 = 64, len = len0, slot = it.slot[0];
    while (true) {
      if (t0 >= len) {
        if (++jj >= gn0) break;
        const bool lo = jj < it.n_inline;
        slot = __builtin_amdgcn_readlane(lo ? slot_lo : slot_hi, jj);
        len = __builtin_amdgcn_readlane(lo ? len_lo : len_hi, jj);
        t0 = 0;
      }
      load_step(kr, vr, slot, t0, len);
      do_step(kr, vr, t0, len);
      t0 += 64;
    }
    for (int g0 = it.cb + 64; g0 < it.ce; g0 += 64) {
      const int gn = min(64, it.ce - g0);
      int my_slot = 0, my_len = 0;
      if (lane < gn) {
        my_slot = P.priv_slot[g0 + lane];
        my_len = P.slot_len[my_slot];
      }
      for (int j = 0; j < gn; ++j) {
        const int sl = __builtin_amdgcn_readlane(my_slot, j);
        const int ln = __builtin_amdgcn_readlane(my_len, j);
        for (int tt = 0; tt < ln; tt += 64) {
          load_step(kr, vr, sl, tt, ln);
          do_step(kr, vr, tt, ln);
        }
      }
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

  auto write_o = [&]() {
    if (tr != 0) return;
    const float inv = 1.f / n;
#pragma unroll
    for (int j = 0; j < EPL; ++j) acc[j] *= inv;
    *reinterpret_cast<uint4*>(static_cast<T*>(P.o) + (static_cast<size_t>(io_row(P.row_map, it.row)) * H + h) * D +
                              sub * EPL) = E::pack(acc);
  };
  if (it.out_part < 0) {
    // fold the row's chunk-first partials (Algorithm 2), then O/n
    if (np <= 64)
      fold_parts_lanes<EPL, 64 / LPT, false>(pidx, P.ws_o, P.o_bytes, P.ws_ml, H, D, h, sub * EPL,
                                             lane, m, n, acc, -1);
    else
      fold_parts<EPL, 64 / LPT, false>(it.part_b, it.part_e, P.parts, P.ws_o, P.o_bytes, P.ws_ml, H,
                                       D, h, sub * EPL, lane, m, n, acc);
    write_o();
    return;
  }
  if (P.cnt) {
    // If every other contributor of the row has already arrived (the usual
    // case: chunk-first items are dispatched first), fold their partials
    // straight into this item's state and finish the row: no partial, no
    // arrival. The counter goes back to zero. This relies on the exchange
    // protocol of device_common.hpp: a count of need - 1, read with a
    // device-scope load, means every other part was visible before it was
    // counted; the branch on it precedes every part load (the compiler
    // fence keeps them there) and those loads are device-scope (DEV = true).
    int32_t* c = P.cnt + static_cast<size_t>(it.row) * H + h;
    int ready = 0;
    if (lane == 0) ready = __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == np - 1;
    if (__shfl(ready, 0)) {
      compiler_fence();
      if (np <= 64)
        fold_parts_lanes<EPL, 64 / LPT, true>(pidx, P.ws_o, P.o_bytes, P.ws_ml, H, D, h, sub * EPL,
                                              lane, m, n, acc, it.out_part);
      else
        fold_parts<EPL, 64 / LPT, true>(it.part_b, it.part_e, P.parts, P.ws_o, P.o_bytes, P.ws_ml, H,
                                        D, h, sub * EPL, lane, m, n, acc, it.out_part);
      if (lane == 0) __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      write_o();
      return;
    }
  }
  if (tr == 0) {
    const __amdgpu_buffer_rsrc_t rs = part_rsrc(P.ws_o, P.o_bytes);
#pragma unroll
    for (int j = 0; j < EPL; j += 4)
      st_dev4(rs, part_off(it.out_part, H, D, h, sub * EPL + j), acc[j], acc[j + 1], acc[j + 2],
              acc[j + 3]);
    if (sub == 0) {
      float* pml = reinterpret_cast<float*>(P.ws_ml + static_cast<size_t>(it.out_part) * H + h);
      st_dev(pml, m);
      st_dev(pml + 1, n);
    }
  }
  if (P.cnt) {
    // partial-writing schedules: the last contributor of the row finishes it
    wait_stores();
    int last = 0;
    if (lane == 0) last = arrive_last(P.cnt + static_cast<size_t>(it.row) * H + h, np);
    if (__shfl(last, 0))
      finish_row<T, D, true>(P.part_ptr, P.parts, P.ws_o, P.o_bytes, P.ws_ml, P.o, P.row_map, H, it.row, h,
                             lane);
  }
}

// ---------------------------------------------------------------------------
// Merge epilogue: rows whose result is spread over several partials.

struct KmgParams {
  void* o;
  const int32_t* row_map;
  const int32_t* mg_rows;
  const int32_t* part_ptr;
  const int32_t* parts;
  const float* ws_o;
  const float2* ws_ml;
  uint32_t o_bytes;
  int H;
};

template <typename T, int D>
__global__ __launch_bounds__(64) void kmg_kernel(KmgParams P) {
  finish_row<T, D, false>(P.part_ptr, P.parts, P.ws_o, P.o_bytes, P.ws_ml, P.o, P.row_map, P.H,
                          P.mg_rows[blockIdx.x],
                          blockIdx.y, threadIdx.x);
}

// ---------------------------------------------------------------------------
// Chunk-first phase on the matrix cores.

struct KcfParams {
  const void* q;
  const void* kpool;
  const void* vpool;
  int64_t ss, hs;  // pool strides of a slot and of a head (elements)
  const int32_t* slot_len;
  const CfSeg* segs;
  const int32_t* seg_slots;
  float* ws_o;
  float2* ws_ml;
  uint32_t o_bytes;  // bytes of the partial-O region at ws_o
  int H;
  int C;
  float qscale;
  // partial-writing schedules only (null otherwise): per (row, head) arrival counters
  // and what the last contributor needs to finish the row
  int32_t* cnt;
  void* o;
  const int32_t* part_ptr;
  const int32_t* parts;
  const int32_t* row_map;  // tree row -> row of q and o (null: tree order)
  int seg_base = 0;        // index in the whole segment list of segs[0]
};

// Partial-writing schedules: after a chunk-first block wrote its partials for
// rows [rb, rb+nrows), count its arrival on each row; the rows for which it
// is the last contributor are finished here (Eqn 2 over the row's partials,
// then O/n) by the whole block at once: each row gets 256/R threads and each
// thread a slice of d, and all loads of a batch of partials are in flight
// together. The rows' partial lists are part of the kernel context, so they
// are requested before the block waits for its own stores; after the
// arrival only the partials themselves are read (one round trip per batch
// instead of a chain of index, maximum and vector loads per row).
constexpr int kFinishBatch = 4;  // partials per batch of the block-wide finish

// The partial list of the row this thread would finish (static context):
// its range is requested once the block's first K/V loads are out
// (finish_range) and its first indices right after the chunk loop
// (finish_ids), so the arrival waits for nothing but the block's own
// partial stores and no load of the block's start waits behind them.
struct FinishList {
  int k0 = 0, k1 = 0;
  int pid[kFinishBatch] = {-1, -1, -1, -1};
};
template <int R>
__device__ __forceinline__ void finish_range(const KcfParams& P, int rb, int nrows, FinishList& f) {
  const int i = static_cast<int>(threadIdx.x) / (256 / R);
  if (P.cnt && i < nrows) {
    f.k0 = P.part_ptr[rb + i];
    f.k1 = P.part_ptr[rb + i + 1];
  }
}
__device__ __forceinline__ void finish_ids(const KcfParams& P, FinishList& f) {
#pragma unroll
  for (int j = 0; j < kFinishBatch; ++j) f.pid[j] = f.k0 + j < f.k1 ? P.parts[f.k0 + j] : -1;
}

template <typename T, int D, int R>
__device__ __forceinline__ void cf_arrive(const KcfParams& P, int rb, int nrows, int h,
                                          float (*red)[R], FinishList fl) {
  constexpr int TPR = 256 / R;   // threads per row
  constexpr int DPT = D / TPR;   // d values per thread
  constexpr int NBF = kFinishBatch;
  static_assert(DPT % 4 == 0 && DPT >= 4, "finish layout");
  const int tid = threadIdx.x;
  const int i = tid / TPR, d0 = (tid % TPR) * DPT;
  const bool mine = i < nrows;
  const int row = rb + i;
  const int k0 = fl.k0, k1 = fl.k1;
  int pid[NBF];
#pragma unroll
  for (int j = 0; j < NBF; ++j) pid[j] = fl.pid[j];
  wait_stores();
  __syncthreads();  // every wavefront's partial stores have completed
  unsigned* flags = reinterpret_cast<unsigned*>(&red[0][0]);
  if (tid < R) {
    int last = 0;
    if (tid < nrows) {
      const int r = rb + tid;
      last = arrive_last(P.cnt + static_cast<size_t>(r) * P.H + h,
                         P.part_ptr[r + 1] - P.part_ptr[r]);
    }
    flags[tid] = last;
  }
  __syncthreads();
  if (!mine || !flags[i]) return;  // no barrier follows
  compiler_fence();
  const int H = P.H;
  const __amdgpu_buffer_rsrc_t rs = part_rsrc(P.ws_o, P.o_bytes);
  float m = kNegBig, n = 0.f, acc[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[e] = 0.f;
  const int p0 = pid[0];  // a finishing row has at least one partial
  for (int kb = k0; kb < k1; kb += NBF) {
    if (kb > k0) {
#pragma unroll
      for (int j = 0; j < NBF; ++j) pid[j] = kb + j < k1 ? P.parts[kb + j] : -1;
    }
    float pm[NBF], pn[NBF];
    float4 pv[NBF][DPT / 4];
#pragma unroll
    for (int j = 0; j < NBF; ++j) {
      const int pk = pid[j] >= 0 ? pid[j] : p0;  // absent: read a valid partial, weight 0
      const float* ml = reinterpret_cast<const float*>(P.ws_ml + static_cast<size_t>(pk) * H + h);
      pm[j] = ld_dev(ml);
      pn[j] = ld_dev(ml + 1);
#pragma unroll
      for (int q = 0; q < DPT / 4; ++q) pv[j][q] = ld_dev4(rs, part_off(pk, H, D, h, d0 + 4 * q));
    }
    float M = m;
#pragma unroll
    for (int j = 0; j < NBF; ++j)
      if (pid[j] >= 0) M = fmaxf(M, pm[j]);
    const float a = fast_exp2(m - M);
    n *= a;
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] *= a;
#pragma unroll
    for (int j = 0; j < NBF; ++j) {
      const float wj = pid[j] >= 0 ? fast_exp2(pm[j] - M) : 0.f;
      n = fmaf(wj, pn[j], n);
#pragma unroll
      for (int q = 0; q < DPT / 4; ++q) {
        acc[4 * q] = fmaf(wj, pv[j][q].x, acc[4 * q]);
        acc[4 * q + 1] = fmaf(wj, pv[j][q].y, acc[4 * q + 1]);
        acc[4 * q + 2] = fmaf(wj, pv[j][q].z, acc[4 * q + 2]);
        acc[4 * q + 3] = fmaf(wj, pv[j][q].w, acc[4 * q + 3]);
      }
    }
    m = M;
  }
  const float inv = 1.f / n;
  T* out = static_cast<T*>(P.o) + (static_cast<size_t>(io_row(P.row_map, row)) * H + h) * D + d0;
#pragma unroll
  for (int e = 0; e < DPT; ++e) out[e] = static_cast<T>(acc[e] * inv);
}

// Lazy reference maximum of the chunk-first softmax (log2 units): P <= 2^8.
constexpr float kLazyMax = 8.f;

// Matrix-core operand layout used below (16x16 output tiles, 64 lanes;
// l16 = lane % 16, g = lane / 16):
//   A (16 x K): lane holds row l16, its K-slice g;   B (K x 16): column l16,
//   K-slice g;   C/D (16 x 16): lane holds rows 4g..4g+3 of column l16.
// Both operands use the same K-slice per lane, so the contraction does not
// depend on how the hardware orders K inside a slice.
template <int D, int NRT, int NCH = 1>
constexpr int kcf_f16_lds_bytes() {
  constexpr int R = 16 * NRT;
  constexpr int NW = 4 * NCH;               // wavefronts
  constexpr int vb = NW * 16 * (D + 16) * 2;  // one V slice per wavefront
  constexpr int ob = NW * R * (D + 4) * 4;    // one merge buffer per wavefront (reuses the slices)
  return (vb > ob ? vb : ob) + 2 * NW * R * 4;
}

// Chunk-first block, fp16. Wavefronts work independently: wavefront w owns
// tokens 16w..16w+15 of every 64-token block of the segment's chunks.
//   S^T = K Q^T: 16x16x32 MFMA, K rows of its 16 tokens as A, the covered q
//     rows as B; the lane then holds S^T[token 4g+i][row l16].
//   online softmax per (wavefront, row): max over its 16 tokens (4 values
//     per lane, then across the four lane groups by shuffles).
//   O^T += V^T P^T: 16x16x16 MFMA whose B operand (lane holds k = 4g..4g+3
//     of column l16) is exactly the layout S^T came out in, so P never leaves
//     the registers; V^T comes from the wavefront's own 16-token V slice in
//     LDS through the transposing ds_read_b64_tr_b16, all d tiles requested
//     before the first of their MFMAs (row stride d+16 halves: the eight rows
//     one half-wavefront reads fall in disjoint banks).
// No barrier inside the chunk loop; the four wavefront states are merged
// once at the end of the segment.
template <int D, int NRT, typename OUT_T = _Float16, int NCH = 1>
__device__ __forceinline__ void kcf_f16_block(const KcfParams& P, int seg, int z, int h, char* lds) {
  constexpr int KS = D / 32;      // 16x16x32 steps over d for S^T
  constexpr int DT = D / 16;      // 16-wide d tiles of O^T (every wavefront holds all)
  constexpr int RS = D + 16;      // V slice row stride (halves)
  constexpr int OS = D + 4;       // merge buffer row stride (floats)
  constexpr int R = 16 * NRT;
  constexpr int NW = 4 * NCH;     // wavefronts: NCH chains of four
  constexpr int VB = NW * 16 * RS * 2;
  constexpr int OB = NW * R * OS * 4;
  constexpr int BIG = VB > OB ? VB : OB;
  constexpr int GPR = D / 8;      // 16-byte granules per token row
  constexpr int TPL = 64 / GPR;   // tokens per wavefront load
  constexpr int NVL = 16 / TPL;   // V loads per lane per block
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wq = w & 3;                                       // token quarter of a block
  const int chain = __builtin_amdgcn_readfirstlane(w >> 2);  // chain (wave-uniform)
  const int l16 = lane & 15, g = lane >> 4;
  _Float16* vw = reinterpret_cast<_Float16*>(lds) + w * 16 * RS;
  float* obuf = reinterpret_cast<float*>(lds);
  float* mbuf = reinterpret_cast<float*>(lds + BIG);  // [NW][R]
  float* nbuf = mbuf + NW * R;                        // [NW][R]

  // The segment's slots sit at a fixed stride, so they are requested with
  // the segment record, in the same round trip (one per lane).
  const CfSeg sg = P.segs[seg];
  const int my_slot = P.seg_slots[(P.seg_base + seg) * kSegSlotStride + lane];
  const int H = P.H, C = P.C;
  const int rb = sg.row_begin + z * R;
  const int nrows = min(R, sg.row_end - rb);
  if (nrows <= 0) return;
  FinishList fl;
  const int nrt = (nrows + 15) / 16;
  const _Float16* q = static_cast<const _Float16*>(P.q);
  const _Float16* kpool = static_cast<const _Float16*>(P.kpool) + h * P.hs;
  const _Float16* vpool = static_cast<const _Float16*>(P.vpool) + h * P.hs;
  const size_t slot_stride = static_cast<size_t>(P.ss);

  // q rows of the block. With two chains (the launch of chunk-first work
  // alone) all of a row's loads go out together after one row-map lookup,
  // with no branches (a lane past the covered rows reads a covered row and
  // keeps zeros), so q, the chunk lengths and the first K/V rows overlap:
  // 0.3-0.9 us less per call on identical prompts. In the fused launch the
  // same change made the call 0.4 us (warm) to 1 us (cold) slower on the
  // bench tree, so there each load stays behind its own row test.
  half8 qf[NRT][KS];
  if constexpr (NCH > 1) {
#pragma unroll
    for (int t = 0; t < NRT; ++t) {
      const int r = 16 * t + l16;
      const _Float16* qp =
          q + (static_cast<size_t>(io_row(P.row_map, rb + min(r, nrows - 1))) * H + h) * D + 8 * g;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const half8 x = *reinterpret_cast<const half8*>(qp + 32 * s);
        qf[t][s] = r < nrows ? x : half8{};
      }
    }
  } else {
#pragma unroll
    for (int t = 0; t < NRT; ++t) {
      const int r = 16 * t + l16;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        if (r < nrows)
          qf[t][s] = *reinterpret_cast<const half8*>(
              q + (static_cast<size_t>(io_row(P.row_map, rb + r)) * H + h) * D + 32 * s + 8 * g);
        else
          qf[t][s] = half8{};
      }
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

  // Segment chunks (at most 64): lane j holds chunk j's slot and length.
  const int my_len = lane < sg.n_chunks ? P.slot_len[my_slot] : 0;
  // Software pipeline: the next block's K rows are requested as soon as the
  // S^T MFMAs have read this block's, and its V rows as soon as this block's
  // V rows are in LDS, so each block's loads overlap the previous block's
  // arithmetic with no extra registers (the fused launch's register count
  // sets every block's occupancy). Every step issues the same loads, so each
  // wait covers only the rows it needs; past the last block a chain
  // re-requests one row of its last block (never used).
  const int ktok = 16 * wq + l16;  // this lane's K row within a block
  const int nch = sg.n_chunks;
  struct Cur {
    int j, t0, slot, len;  // block = rows t0 .. t0 + 63 of the segment's chunk j
  };
  auto valid = [&](const Cur& c) { return c.j < nch; };
  auto step = [&](Cur c) {
    c.t0 += 64;
    if (c.t0 >= c.len) {
      c.t0 = 0;
      c.j += NCH;
      if (c.j < nch) {
        c.slot = __builtin_amdgcn_readlane(my_slot, c.j);
        c.len = __builtin_amdgcn_readlane(my_len, c.j);
      }
    }
    return c;
  };
  // past the end: one row of block c (the rest of the block reads as zeros)
  auto dummy = [&](Cur c) {
    c.t0 = c.len - 1;
    return c;
  };
  // K and V rows of block c go through a buffer descriptor that spans
  // exactly the block's valid rows: its base (slot, first row) is
  // wave-uniform, so the address arithmetic is scalar and each lane's byte
  // offset is the same in every block, and rows past the valid length read
  // as zeros (the descriptor's range check; their scores are masked below,
  // so they add nothing).
  auto rows_rsrc = [&](const _Float16* pool, const Cur& c) {
    const int slot = __builtin_amdgcn_readfirstlane(c.slot);
    const int t0 = __builtin_amdgcn_readfirstlane(c.t0);
    const int ntb = min(64, __builtin_amdgcn_readfirstlane(c.len) - t0);
    return __builtin_amdgcn_make_buffer_rsrc(
        const_cast<_Float16*>(pool + slot * slot_stride + static_cast<size_t>(t0) * D), 0, ntb * D * 2,
        kRsrcWord3);
  };
  const int ko = (ktok * D + 8 * g) * 2;  // this lane's K granule (s = 0), bytes
  int vo[NVL];                            // this lane's V granules, bytes
#pragma unroll
  for (int i = 0; i < NVL; ++i) vo[i] = ((16 * wq + lane / GPR + TPL * i) * D + (lane % GPR) * 8) * 2;
  auto load_k = [&](half8 (&kf)[KS], const Cur& c) {
    const __amdgpu_buffer_rsrc_t r = rows_rsrc(kpool, c);
#pragma unroll
    for (int s = 0; s < KS; ++s)
      kf[s] = __builtin_bit_cast(half8, __builtin_amdgcn_raw_buffer_load_b128(r, ko + 64 * s, 0, 0));
  };
  auto load_v = [&](uint4 (&vr)[NVL], const Cur& c) {
    const __amdgpu_buffer_rsrc_t r = rows_rsrc(vpool, c);
#pragma unroll
    for (int i = 0; i < NVL; ++i)
      vr[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, vo[i], 0, 0));
  };
  // block `cur` from the register set (kf, vr); then block `req` into it
  auto body = [&](half8 (&kf)[KS], uint4 (&vr)[NVL], const Cur& cur, const Cur& req) {
    const int nt = min(64, cur.len - cur.t0);
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
    load_k(kf, req);
    // Online softmax with a lazy reference maximum: a row's reference m_run
    // moves only when the block's maximum exceeds it by more than kLazyMax
    // (log2 units), so P = exp2(S - m_run) <= 2^kLazyMax (exactly
    // representable range of fp16, same relative precision), and the O
    // accumulators (in AGPRs: a rescale is a read, a multiply and a write
    // per register) are rescaled only in the blocks where some row's
    // reference moved (wave-uniform test), not in every block. Any reference
    // gives the same O / n; the partial carries the reference it used.
    half4 ph[NRT];
    float alpha[NRT];
    bool moved = false;
#pragma unroll
    for (int t = 0; t < NRT; ++t) {
      float lmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = 16 * wq + 4 * g + i;
        const float x = tok < nt ? sacc[t][i] * P.qscale : -INFINITY;
        sacc[t][i] = x;
        lmax = fmaxf(lmax, x);
      }
      lmax = rows4_max(lmax);
      const float mn = lmax > m_run[t] + kLazyMax ? lmax : m_run[t];
      alpha[t] = fast_exp2(m_run[t] - mn);
      moved |= mn != m_run[t];
      m_run[t] = mn;
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ph[t][i] = static_cast<_Float16>(fast_exp2(sacc[t][i] - mn));
        ps += static_cast<float>(ph[t][i]);
      }
      n_part[t] = n_part[t] * alpha[t] + ps;
    }
    // this wavefront's 16 V rows -> its LDS slice (its previous reads of the
    // slice precede these writes in program order)
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int tl = lane / GPR + TPL * i;
      uint2* dst = reinterpret_cast<uint2*>(vw + tl * RS + (lane % GPR) * 8);
      dst[0] = make_uint2(vr[i].x, vr[i].y);
      dst[1] = make_uint2(vr[i].z, vr[i].w);
    }
    load_v(vr, req);
    if (__any(moved)) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int t = 0; t < NRT; ++t) acc[dt][t] *= alpha[t];
    }
    half4 va[DT];  // lane: tokens 4g..4g+3 of column 16dt + l16
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) va[dt] = lds_read_tr16(vw + (4 * g + (l16 >> 2)) * RS + 16 * dt + 4 * (l16 & 3));
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        if (t < nrt) acc[dt][t] = __builtin_amdgcn_mfma_f32_16x16x16f16(va[dt], ph[t], acc[dt][t], 0, 0, 0);
      }
    }
  };
  // The first block's rows go out before the first chunk's length is
  // known, as if it were full (a range over the slot's first min(C, 64)
  // rows: in bounds, but rows past the length may hold anything, even NaN);
  // a shorter chunk is requested again with its own range, so those rows
  // read as zeros. Chain k takes chunks k, k + NCH, ... (a chain with no
  // chunk skips the loop and merges an empty state).
  const int cm = min(C, 64);
  Cur cur{chain, 0, __builtin_amdgcn_readlane(my_slot, chain), cm};
  half8 kA[KS];
  uint4 vA[NVL];
  const bool work = chain < nch;
  if (work) {
    load_k(kA, cur);
    load_v(vA, cur);
  }
  finish_range<R>(P, rb, nrows, fl);
  cur.len = __builtin_amdgcn_readlane(my_len, chain);
  if (work && cur.len < cm) {  // uniform; rare
    load_k(kA, cur);
    load_v(vA, cur);
  }
  while (work) {
    const Cur nxt = step(cur);
    const bool more = valid(nxt);
    body(kA, vA, cur, more ? nxt : dummy(cur));
    if (!more) break;
    cur = nxt;
  }

  finish_ids(P, fl);
  // Merge the wavefront states per row: common max, rescaled sums.
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    float ns = n_part[t];
    ns += __shfl_xor(ns, 16);
    ns += __shfl_xor(ns, 32);
    if (g == 0) {
      mbuf[w * R + 16 * t + l16] = m_run[t];
      nbuf[w * R + 16 * t + l16] = ns;
    }
  }
  __syncthreads();  // all wavefronts are past their loops: the slices are free
  float scale[NRT], Mrow[NRT], Nrow[NRT];
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    const int r = 16 * t + l16;
    float M = kNegBig;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, mbuf[ww * R + r]);
    float N = 0.f;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) N += nbuf[ww * R + r] * fast_exp2(mbuf[ww * R + r] - M);
    scale[t] = fast_exp2(m_run[t] - M);
    Mrow[t] = M;
    Nrow[t] = N;
  }
  // every wavefront parks its rescaled O^T in its own buffer ([row][d], one
  // 16-byte write per tile); the partial stores below add them up
  {
    float* mine = obuf + w * (R * OS);
#pragma unroll
    for (int t = 0; t < NRT; ++t) {
      if (t < nrt) {
        const int r = 16 * t + l16;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<floatx4*>(mine + r * OS + 16 * dt + 4 * g) = acc[dt][t] * scale[t];
      }
    }
  }
  __syncthreads();
  // write the segment's partial (O, m, n) for every covered row
  const size_t pbase = static_cast<size_t>(sg.part_base + (rb - sg.row_begin));
  const bool fold = sg.pad0 != 0;
  if (fold) {
    // serial reduction: fold into the row's accumulator (Eqn 2), which an
    // earlier launch wrote; per-row factors go through mbuf / nbuf (free now)
    if (w == 0 && g == 0) {
#pragma unroll
      for (int t = 0; t < NRT; ++t) {
        const int r = 16 * t + l16;
        if (r < nrows) {
          const float* pml = reinterpret_cast<const float*>(P.ws_ml + (pbase + r) * H + h);
          const float mp = ld_dev(pml), np = ld_dev(pml + 1);
          const float mx = fmaxf(Mrow[t], mp);
          const float x = fast_exp2(Mrow[t] - mx), y = fast_exp2(mp - mx);
          mbuf[r] = x;
          nbuf[r] = y;
          Mrow[t] = mx;
          Nrow[t] = x * Nrow[t] + y * np;
        }
      }
    }
    __syncthreads();
  }
  {
    const __amdgpu_buffer_rsrc_t rs = part_rsrc(P.ws_o, P.o_bytes);
    for (int e = tid; e < nrows * (D / 4); e += 256 * NCH) {
      const int r = e / (D / 4), d = 4 * (e % (D / 4));
      float4 v = *reinterpret_cast<const float4*>(obuf + r * OS + d);
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) {
        const float4 u = *reinterpret_cast<const float4*>(obuf + ww * (R * OS) + r * OS + d);
        v = make_float4(v.x + u.x, v.y + u.y, v.z + u.z, v.w + u.w);
      }
      const uint32_t off = part_off(static_cast<int>(pbase) + r, H, D, h, d);
      if (fold) {
        const float4 pv = ld_dev4(rs, off);
        const float x = mbuf[r], y = nbuf[r];
        v = make_float4(x * v.x + y * pv.x, x * v.y + y * pv.y, x * v.z + y * pv.z,
                        x * v.w + y * pv.w);
      }
      st_dev4(rs, off, v.x, v.y, v.z, v.w);
    }
  }
  if (w == 0 && g == 0) {
#pragma unroll
    for (int t = 0; t < NRT; ++t) {
      const int r = 16 * t + l16;
      if (r < nrows) {
        float* pml = reinterpret_cast<float*>(P.ws_ml + (pbase + r) * H + h);
        st_dev(pml, Mrow[t]);
        st_dev(pml + 1, Nrow[t]);
      }
    }
  }
  if (P.cnt) cf_arrive<OUT_T, D, R>(P, rb, nrows, h, reinterpret_cast<float (*)[R]>(mbuf), fl);
}

// fp32 chunk-first on the 16x16x4 fp32 matrix-core op (operands are single
// floats: A row l16, k = g; B column l16, k = g), with the earlier schedule:
// wavefront w computes S^T for tokens 16w..16w+15 of each 64-token block and
// O^T for the d columns [w*D/4, (w+1)*D/4), so P = exp2(S - m) goes through
// LDS ([row][token]) and V is staged in LDS ([token][d], rows padded by one
// element), with barriers inside the chunk loop.
template <int D, int NRT>
constexpr int kcf_f32_lds_bytes() {
  return 64 * (D + 1) * 4 + 16 * NRT * (64 + 1) * 4 + 4 * 16 * NRT * 4;
}

template <int D, int NRT, typename OUT_T = float>
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
  FinishList fl;
  finish_range<R>(P, rb, nrows, fl);
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
    const size_t base = static_cast<size_t>(slot) * P.ss + h * P.hs;
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
            const float b = r < nrows ? q[(static_cast<size_t>(io_row(P.row_map, rb + r)) * H + h) * D + 4 * s + g] : 0.f;
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

  finish_ids(P, fl);
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    float ns = n_part[t];
    ns += __shfl_xor(ns, 16);
    ns += __shfl_xor(ns, 32);
    if (g == 0) red[w][16 * t + l16] = ns;
  }
  __syncthreads();
  // m_run is the same in every wavefront (block-wide maxima), so each lane
  // derives its row's fold factors itself
  const bool fold = sg.pad0 != 0;
#pragma unroll
  for (int t = 0; t < NRT; ++t) {
    const int r = 16 * t + l16;
    if (r < nrows) {
      const size_t p = static_cast<size_t>(sg.part_base + (rb - sg.row_begin) + r);
      const __amdgpu_buffer_rsrc_t rs = part_rsrc(P.ws_o, P.o_bytes);
      float* pml = reinterpret_cast<float*>(P.ws_ml + p * H + h);
      float m = m_run[t], n = red[0][r] + red[1][r] + red[2][r] + red[3][r];
      float x = 1.f, y = 0.f;
      if (fold) {
        // serial reduction: fold into the row's accumulator (Eqn 2)
        const float mp = ld_dev(pml), np = ld_dev(pml + 1);
        const float mx = fmaxf(m, mp);
        x = fast_exp2(m - mx);
        y = fast_exp2(mp - mx);
        m = mx;
        n = x * n + y * np;
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        floatx4 v = acc[dt][t];
        const uint32_t off = part_off(static_cast<int>(p), H, D, h, w * (D / 4) + 16 * dt + 4 * g);
        if (fold) {
          const float4 pv = ld_dev4(rs, off);
          v = floatx4{x * v[0] + y * pv.x, x * v[1] + y * pv.y, x * v[2] + y * pv.z,
                      x * v[3] + y * pv.w};
        }
        st_dev4(rs, off, v[0], v[1], v[2], v[3]);
      }
      if (w == 0 && g == 0) {
        st_dev(pml, m);
        st_dev(pml + 1, n);
      }
    }
  }
  if (P.cnt) cf_arrive<OUT_T, D, R>(P, rb, nrows, h, red, fl);
}

// ---------------------------------------------------------------------------
// K/V copies for tree operations.

struct KvJobBatch {
  int32_t n;
  KvJob job[kKvJobsPerLaunch];
};

__global__ __launch_bounds__(256) void kkv_kernel(KvJobBatch b, const char* k, const char* v,
                                                  char* kpool, char* vpool, int32_t* slot_len,
                                                  int H, int row_bytes, int64_t ss_bytes,
                                                  int64_t hs_bytes) {
  const KvJob j = b.job[blockIdx.x];
  const int h = blockIdx.y;
  if (j.kind != 2) {
    const int units = row_bytes / 16;
    const size_t dst = static_cast<size_t>(j.dst_slot) * ss_bytes + h * hs_bytes +
                       static_cast<size_t>(j.dst_pos) * row_bytes;
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
      src = static_cast<size_t>(j.src) * ss_bytes + h * hs_bytes +
            static_cast<size_t>(j.src_pos) * row_bytes;
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

// Schedules. 0 sequential: chunk-first launch, then a sequence-first launch
// whose items fold the finished chunk-first partials themselves (the merge
// epilogue only finishes split rows). 1 fused: one launch, blocks [0, n_cf)
// run chunk-first items (dispatched first), the rest sequence-first items;
// every item writes a partial and the merge epilogue finishes the rows.
// 2 fused with in-kernel merge: as 1, but every item counts its arrival on
// its rows and the last contributor of a row finishes it. 3 concurrent: the
// chunk-first kernel on a side stream, the sequence-first kernel on the
// caller's stream at the same time, rows finished as in 2.
struct TppParams {
  KcfParams cf;
  KsfParams sf;
  int n_cf;        // chunk-first blocks: n_segs * zb * H
  int zb;          // row blocks per segment
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
  const int b = static_cast<int>(blockIdx.x);
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

// Chunk-first work alone (no sequence-first item in the call, e.g. identical
// sequences): 16-row blocks of eight wavefronts, two chains of four that take
// alternate chunks of the segment, so each block keeps twice the loads in
// flight and the chains' states are merged once at the end. Measured on
// Table 3's all-shared cells against one chain with a two-deep prefetch
// (same) and four chains (slower: more fixed cost per chain).
constexpr int kDeepChains = 2;
template <int D>
__global__ __launch_bounds__(256 * kDeepChains) void kcf_deep_kernel(KcfParams P, int zb) {
  __shared__ __attribute__((aligned(16))) char lds[kcf_f16_lds_bytes<D, 1, kDeepChains>()];
  const int b = static_cast<int>(blockIdx.x);
  const int h = b % P.H;
  const int rest = b / P.H;
  kcf_f16_block<D, 1, _Float16, kDeepChains>(P, rest / zb, rest % zb, h, lds);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void ksf_kernel(KsfParams P) {
  __shared__ __attribute__((aligned(16))) char lds[ksf_lds_bytes<T, D>()];
  const int b = static_cast<int>(blockIdx.x);
  ksf_block<T, D>(P, b / P.H, b % P.H, lds);
}

template <typename T, int D, int NRT>
hipError_t launch_phases(const TppParams& P, int n_sf, int schedule, int mask, hipStream_t s,
                         const SideStream& side, const int32_t* group_ptr, int n_groups) {
  const bool both = (mask & 3) == 3;
  if ((schedule == 1 || schedule == 2) && both) {
    // the fused launch always takes 16-row chunk-first blocks
    if constexpr (NRT == 1) {
      if constexpr (sizeof(T) == 2) {
        if (n_sf == 0) {  // chunk-first work alone
          if (P.n_cf > 0) kcf_deep_kernel<D><<<P.n_cf, 256 * kDeepChains, 0, s>>>(P.cf, P.zb);
          return hipSuccess;
        }
      }
      const int grid = P.n_cf + n_sf;
      if (grid > 0) tpp_kernel<T, D, NRT><<<grid, 256, 0, s>>>(P);
      return hipSuccess;
    } else {
      return hipErrorInvalidValue;
    }
  }
  if (schedule == 3 && both && P.n_cf > 0 && n_sf > 0) {
    // chunk-first on the side stream, sequence-first on the caller's stream,
    // concurrently; the caller's stream then waits for the side stream
    hipError_t e;
    if ((e = hipEventRecord(side.fork, s)) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(side.stream, side.fork, 0)) != hipSuccess) return e;
    kcf_kernel<T, D, NRT><<<P.n_cf, 256, 0, side.stream>>>(P.cf, P.zb);
    if ((e = hipEventRecord(side.join, side.stream)) != hipSuccess) return e;
    ksf_kernel<T, D><<<n_sf, 256, 0, s>>>(P.sf);
    return hipStreamWaitEvent(s, side.join, 0);
  }
  // phases one after another on the caller's stream; arrival counting only
  // when this is the complete attention of a counting schedule
  KcfParams cf = P.cf;
  KsfParams sf = P.sf;
  if (!both) {
    cf.cnt = nullptr;
    sf.cnt = nullptr;
  }
  if (schedule == 4) {
    // serial reduction: the g-th launch runs every row's g-th chunk-first
    // segment, which folds into the row's accumulator; the kernel boundary
    // orders the writers of each row, so no row has two at once
    if ((mask & 1) && P.n_cf > 0) {
      for (int gi = 0; gi < n_groups; ++gi) {
        KcfParams g = cf;
        g.segs = cf.segs + group_ptr[gi];
        g.seg_base = group_ptr[gi];
        const int nb = (group_ptr[gi + 1] - group_ptr[gi]) * P.zb * cf.H;
        if (nb > 0) kcf_kernel<T, D, NRT><<<nb, 256, 0, s>>>(g, P.zb);
      }
    }
  } else if ((mask & 1) && P.n_cf > 0) {
    kcf_kernel<T, D, NRT><<<P.n_cf, 256, 0, s>>>(cf, P.zb);
  }
  if ((mask & 2) && n_sf > 0) ksf_kernel<T, D><<<n_sf, 256, 0, s>>>(sf);
  return hipSuccess;
}

template <typename T, int D>
hipError_t launch_all(const AttnArgs& a, const DevWork& w, hipStream_t s, int mask,
                      const SideStream& side) {
  TppParams P;
  const bool counting = w.schedule == 2 || w.schedule == 3;  // the last contributor finishes each row
  P.cf = KcfParams{a.q, a.kpool, a.vpool, a.ss, a.hs, a.slot_len, w.segs, w.seg_slots, a.ws_o,
                   reinterpret_cast<float2*>(a.ws_ml), a.ws_o_bytes, a.H, a.C, a.qscale,
                   counting ? a.cnt : nullptr, a.o, w.part_ptr, w.parts, a.row_map};
  P.sf = KsfParams{a.q, a.o, a.kpool, a.vpool, a.ss, a.hs, a.slot_len, w.items, w.priv_slot, w.part_ptr,
                   w.parts, a.ws_o, reinterpret_cast<float2*>(a.ws_ml), a.ws_o_bytes, a.H, a.C,
                   a.qscale, counting ? a.cnt : nullptr, a.row_map};
  // At most 16 or 32 covered rows per chunk-first block; wider runs take
  // several row blocks, which re-read the chunk. Their block indices differ
  // by a multiple of H, so for H a multiple of 8 they land on the same XCD
  // (blocks go to XCDs round-robin) and the re-reads hit that XCD's L2.
  // The fused launch carries the chunk-first path's registers into every
  // block, so there chunk-first blocks take 16 rows; alone they take 32.
  const int rows = w.max_seg_rows;
  const bool fused = (w.schedule == 1 || w.schedule == 2) && (mask & 3) == 3;
  const int nrt = rows <= 16 || fused ? 1 : 2;
  P.zb = rows > 0 ? (rows + 16 * nrt - 1) / (16 * nrt) : 1;
  P.n_cf = w.n_segs * P.zb * a.H;
  const int n_sf = w.n_items * a.H;
  hipError_t e;
  if (nrt == 1) e = launch_phases<T, D, 1>(P, n_sf, w.schedule, mask, s, side, w.seg_group_ptr, w.n_seg_groups);
  else e = launch_phases<T, D, 2>(P, n_sf, w.schedule, mask, s, side, w.seg_group_ptr, w.n_seg_groups);
  if (e != hipSuccess) return e;
  // Partial-writing schedules finish their rows inside the kernels; the merge
  // epilogue runs in the sequential schedule (split rows) or on its own.
  const bool self_finished = counting && (mask & 3) == 3;
  if ((mask & 4) && w.n_mg > 0 && !self_finished) {
    KmgParams M{a.o, a.row_map, w.mg_rows, w.part_ptr, w.parts, a.ws_o, reinterpret_cast<const float2*>(a.ws_ml),
                a.ws_o_bytes, a.H};
    kmg_kernel<T, D><<<dim3(w.n_mg, a.H), 64, 0, s>>>(M);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, const DevWork& w, hipStream_t s, int mask,
                            const SideStream& side) {
  if (a.dtype == 0) {
    if (a.D == 128) return launch_all<_Float16, 128>(a, w, s, mask, side);
    if (a.D == 64) return launch_all<_Float16, 64>(a, w, s, mask, side);
  } else {
    if (a.D == 128) return launch_all<float, 128>(a, w, s, mask, side);
    if (a.D == 64) return launch_all<float, 64>(a, w, s, mask, side);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_kv_jobs(const KvJob* jobs, int n, int dtype, int H, int D, int C, int64_t ss,
                          int64_t hs, const void* k, const void* v, void* kpool, void* vpool,
                          int32_t* slot_len, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  if (n > kKvJobsPerLaunch) return hipErrorInvalidValue;
  KvJobBatch b;
  b.n = n;
  for (int i = 0; i < n; ++i) b.job[i] = jobs[i];
  const int row_bytes = D * (dtype == 0 ? 2 : 4);
  const int64_t es = dtype == 0 ? 2 : 4;
  (void)C;
  kkv_kernel<<<dim3(n, H), 256, 0, stream>>>(b, static_cast<const char*>(k),
                                             static_cast<const char*>(v), static_cast<char*>(kpool),
                                             static_cast<char*>(vpool), slot_len, H, row_bytes,
                                             ss * es, hs * es);
  return hipGetLastError();
}

}  // namespace ca
