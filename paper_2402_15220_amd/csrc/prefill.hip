// gfx950 (MI355X) prefill attention with prefix reuse over the prefix-tree,
// chunked KV cache of ChunkAttention (arXiv 2402.15220, Section 3.2,
// prefill paragraph).
#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

#include "device_common.hpp"
#include "kernels.hpp"

namespace ca {
namespace {

// slack of the softmax reference maximum, in log2 units
constexpr float kPfLazyMax = 8.f;

// Prefill with prefix reuse (Section 3.2, prefill paragraph): once a joining
// sequence's unmatched suffix has been written into the tree, its n_q
// trailing tokens attend causally to the sequence's whole K/V, read chunk by
// chunk along the root-to-leaf path. Query i sits at position
// L - n_q + i and sees positions 0..L - n_q + i.
//
// One block per (64 queries, head), NGRP groups of WPG wavefronts. The
// work is a list of units of TOK consecutive rows of one chunk (a chunk of
// up to c tokens is ceil(c / TOK) units); group k takes units k, k+NGRP, ...
// Each group has two LDS tiles: while it computes one unit from one tile,
// the next unit is written into the other tile and the one after is loading
// into registers, so one barrier per step suffices. Inside a group,
// wavefront w owns QT = 4/WPG tiles of 16 queries and every token of the
// group's units; K and V are staged as [token][d], once for all 64 queries,
// and each K or V element read from LDS feeds QT matrix-core ops.
//   S^T = K Q^T  (16x16x32 MFMA: K rows from LDS as A, the wavefront's q rows
//                 as B, held in registers for the whole call);
//   causal and chunk-length mask where a unit needs one, online softmax per
//   query row (base 2, scale folded into the exponent, a lazy reference
//   maximum; the row sums of P on the matrix cores);
//   O^T += V^T P^T (16x16x32 MFMA: V^T read from LDS with the transposing
//                 ds_read_b64_tr_b16 as A, P^T straight from the S^T
//                 accumulators of two token tiles as B).
// At the end the groups' states (m, n, O) are folded (Eqn 2) through LDS
// and group 0 writes o = O / n.
// When the query tiles alone would leave most compute units idle (a short
// join over a long path), each tile's units are cut into n_split contiguous
// parts run by separate blocks: every part writes its (m, n, O) with
// device-scope stores and counts its arrival, and the last part to arrive
// folds all of them (Eqn 2) and writes o; no block waits for another.
struct KpfParams {
  const _Float16* q;            // [n_q][H][D]
  _Float16* o;                  // [n_q][H][D]
  const _Float16* kpool;
  const _Float16* vpool;
  int64_t ss, hs;               // pool strides of a slot and of a head (elements)
  int n_chunks;                 // chunk_slot [n_chunks] path slots root -> leaf, chunk_start
                                // [n_chunks + 1] first position of each chunk (last = L):
                                // kernel arguments of their own
  int n_q;
  int H;
  int C;
  float qscale;                 // softmax scale * log2(e)
  int n_split;                  // key-range parts per (query tile, head); 1: none
  float* ws;                    // n_split > 1: one partial per part, [tile][part] of
                                // kpf_part_floats<D>() floats: O [64][D], then m [64], n [64]
  int32_t* cnt;                 // n_split > 1: arrival counter per tile, zero between launches
  uint32_t ws_bytes;            // bytes of ws (below 4 GiB: 32-bit buffer offsets)
};

// floats of one partial: unnormalised O of 64 query rows, their maxima and sums
template <int D>
constexpr int kpf_part_floats() { return 64 * D + 2 * 64; }
static_assert(prefill_part_bytes(128) == kpf_part_floats<128>() * 4 &&
                  prefill_part_bytes(64) == kpf_part_floats<64>() * 4,
              "partial size shared with the host");

template <int D>
constexpr int kpf_k_stride() { return D + 8; }
template <int D>
constexpr int kpf_v_stride() { return D + 16; }

template <int D, int TOK>
constexpr int kpf_tile_bytes() { return TOK * (kpf_k_stride<D>() + kpf_v_stride<D>()) * 2; }

// A short path travels inside the kernel arguments (no upload before the
// launch); NI is its capacity.
template <int NI>
struct KpfPath {
  int32_t slot[NI];
  int32_t start[NI + 1];
};

// Work unit: TOK consecutive rows of one chunk (a chunk of up to c tokens
// has ceil(c / TOK) units). NI > 0: the path comes in `path` (at most NI
// chunks); NI == 0: in the device arrays cslot / cstart.
template <int D, int NGRP, int WPG, int TOK, int NI>
__global__ __launch_bounds__(64 * WPG * NGRP) void kpf_kernel(KpfParams P,
                                                              const int32_t* __restrict__ cslot,
                                                              const int32_t* __restrict__ cstart,
                                                              const KpfPath<(NI > 0 ? NI : 1)> path) {
  constexpr int QT = 4 / WPG;       // 16-query tiles per wavefront
  constexpr int GT = 64 * WPG;      // threads per group
  constexpr int KS = D / 32;        // 16x16x32 steps over d
  constexpr int DT = D / 16;        // 16-wide d tiles of O^T
  constexpr int NG = D / 8;         // 16-byte granules per token row
  constexpr int GPT = TOK * NG / GT;// granules of K (and of V) per thread per unit
  constexpr int JT = TOK / 16;      // 16-token tiles of S^T per unit
  constexpr int PV = TOK / 32;      // 32-token steps of O^T per unit
  constexpr int KST = kpf_k_stride<D>();
  constexpr int VST = kpf_v_stride<D>();
  constexpr int TB = kpf_tile_bytes<D, TOK>();
  constexpr int OST = D + 4;         // merge buffer row stride (floats): rows start 4 banks apart
  static_assert(WPG * QT == 4, "64 queries per block");
  static_assert(TOK % 32 == 0 && TOK <= 64 && GPT * GT == TOK * NG, "unit shape");
  static_assert(2 * TB * NGRP <= 160 * 1024, "two LDS tiles per group");
  static_assert(NGRP == 1 || 2 * TB * NGRP >= (NGRP - 1) * 64 * (OST + 2) * 4, "merge buffer");
  __shared__ __attribute__((aligned(16))) char lds[2 * TB * NGRP];
  // Chunk j's slot, first position and end. A path of up to 64 chunks keeps
  // chunk j's three values in lane j and reads them with v_readlane, so the
  // unit loop has no memory wait for them (a scalar load's wait would also
  // drain the wavefront's LDS operations); longer paths read the kernel
  // arguments or the device arrays through the scalar cache.
  constexpr bool kLane = NI > 0 && NI <= 64;
  int lane_slot = 0, lane_start = 0x7fffffff, lane_end = 0;
  if constexpr (kLane) {
    const int l = threadIdx.x & 63;
    if (l < P.n_chunks) {
      lane_slot = path.slot[l];
      lane_start = path.start[l];
      lane_end = path.start[l + 1];
    }
  }
  auto chunk_slot = [&](int j) -> int {
    if constexpr (kLane) return __builtin_amdgcn_readlane(lane_slot, j);
    else if constexpr (NI > 0) return path.slot[j];
    else return cslot[j];
  };
  auto chunk_start = [&](int j) -> int {
    if constexpr (kLane) return __builtin_amdgcn_readlane(lane_start, j);
    else if constexpr (NI > 0) return path.start[j];
    else return cstart[j];
  };
  auto chunk_end = [&](int j) -> int {
    if constexpr (kLane) return __builtin_amdgcn_readlane(lane_end, j);
    else if constexpr (NI > 0) return path.start[j + 1];
    else return cstart[j + 1];
  };

  const int tid = threadIdx.x, lane = tid & 63;
  const int grp = __builtin_amdgcn_readfirstlane((tid >> 6) / WPG);  // uniform: unit indices stay scalar
  const int w = (tid >> 6) % WPG;   // wavefront inside the group
  const int gtid = tid % GT;        // thread index inside the group
  const int l16 = lane & 15, g = lane >> 4;
  // the group's two tiles: tile b holds K rows then V rows
  auto tile_k = [&](int b) { return reinterpret_cast<_Float16*>(lds + (2 * grp + b) * TB); };
  // XCD-aware order: blocks go to the eight XCDs round-robin, so block b
  // runs on XCD b % 8; the (tile, part) pairs (tiles head-major, the parts
  // of a tile adjacent) are split into eight contiguous ranges, one per XCD,
  // and every query tile of a head reads that head's chunks through the
  // same L2.
  const int H = P.H, n_q = P.n_q;
  const int n_qt = (n_q + 63) / 64;
  const int per_xcd = static_cast<int>(gridDim.x) / 8;
  const int v = static_cast<int>(blockIdx.x % 8) * per_xcd + static_cast<int>(blockIdx.x / 8);
  const int S = P.n_split;
  if (v >= n_qt * H * S) return;
  const int tix = v / S, part = v % S;   // the parts of a tile are neighbours (same XCD)
  const int h = tix / n_qt;
  const int q0 = (tix % n_qt) * 64;                            // first query of the tile
  // this lane's query row of tile t and its q fragments, requested before
  // anything waits for the chunk table, so the two round trips overlap (and
  // the first unit's loads overlap q's)
  int qi[QT];
  half8 qf[QT][KS];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    qi[t] = q0 + 16 * (QT * w + t) + l16;
    const int qr = min(qi[t], n_q - 1);  // rows past n_q load a valid row (never written)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      qf[t][s] = *reinterpret_cast<const half8*>(P.q + (static_cast<size_t>(qr) * H + h) * D + 32 * s + 8 * g);
  }
  const int L = chunk_end(P.n_chunks - 1);
  const int pos_last = L - n_q + min(q0 + 63, n_q - 1);        // last position of the tile
  const int pos_first = L - n_q + q0;                          // first position of the tile
  const size_t slot_stride = static_cast<size_t>(P.ss);
  const _Float16* kbase = P.kpool + h * P.hs;
  const _Float16* vbase = P.vpool + h * P.hs;
  const int upc = (P.C + TOK - 1) / TOK;                       // units per chunk

  // this lane's query positions
  int pos[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) pos[t] = L - n_q + qi[t];
  // m_run: reference maximum per query row; nacc: the row's sum of P,
  // accumulated on the matrix cores (every row of the 16x16 product holds it)
  float m_run[QT];
  floatx4 acc[QT][DT], nacc[QT];
  const half8 ones8 = {1, 1, 1, 1, 1, 1, 1, 1};
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    m_run[t] = kNegBig;
    nacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[t][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  // Chunks the tile needs: those starting at or before its last position
  // (starts ascend); 64 starts per load, one per lane.
  const int nc = P.n_chunks;
  int n_ch = 0;
  if constexpr (kLane) {
    n_ch = __popcll(__ballot(lane_start <= pos_last));
  } else {
    for (int b = 0; b < nc; b += 64) {
      const int st = b + lane < nc ? chunk_start(b + lane) : 0x7fffffff;
      const unsigned long long m = __ballot(st <= pos_last);
      n_ch += __popcll(m);
      if (m != ~0ull) break;
    }
  }
  const int n_units = n_ch * upc;
  // this block's part of the tile's units
  const int u_lo = static_cast<int>(static_cast<int64_t>(n_units) * part / S);
  const int u_hi = static_cast<int>(static_cast<int64_t>(n_units) * (part + 1) / S);
  // unit u is rows r0 .. r0 + TOK - 1 of chunk j (no division when every
  // chunk is one unit; uniform)
  auto unit_pos = [&](int u, int& j, int& r0) {
    if (upc == 1) {
      j = u;
      r0 = 0;
    } else {
      j = u / upc;
      r0 = TOK * (u - j * upc);
    }
  };
  // Past the end the registers reload the last unit: every step issues the
  // same loads, so the wait before each LDS write covers exactly the
  // registers it needs on every path.
  u32x4 kr[GPT], vr[GPT];
  // K and V rows of a unit go through buffer descriptors that span exactly
  // the unit's valid rows: the base (slot, first row) is wave-uniform, so
  // the address arithmetic is scalar and each lane's byte offset is the same
  // in every step (granule e = gtid + GT*u2 is row e / (D/8), 16-byte column
  // e % (D/8): coalesced rows); rows past the chunk's length read as zeros
  // (their scores are masked, and zero V rows add nothing). 0.9 us less on a
  // 512-token join than per-lane addresses clamped to the chunk.
  int goff[GPT];
#pragma unroll
  for (int u2 = 0; u2 < GPT; ++u2) {
    const int e = gtid + GT * u2;
    goff[u2] = ((e / NG) * D + (e % NG) * 8) * 2;
  }
  auto issue = [&](int u) {
    int j, r0;
    unit_pos(min(u, u_hi - 1), j, r0);
    const int slot = __builtin_amdgcn_readfirstlane(chunk_slot(j));
    // a unit past a short chunk's end (chunks longer than TOK count
    // ceil(c / TOK) units each) gets an empty range: its loads read zeros
    // max(m, 0) written as a scalar instruction: as plain code the compiler
    // turns the clamp into a vector median-of-three, and the descriptor built
    // from a vector register then costs a per-lane loop around every load
    const int m = min(TOK, chunk_end(j) - chunk_start(j) - r0);
    int rows;
    asm("s_max_i32 %0, %1, 0" : "=s"(rows) : "s"(m));
    const size_t base = static_cast<size_t>(slot) * slot_stride + static_cast<size_t>(r0) * D;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<_Float16*>(kbase + base), 0, rows * D * 2, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<_Float16*>(vbase + base), 0, rows * D * 2, kRsrcWord3);
#pragma unroll
    for (int u2 = 0; u2 < GPT; ++u2) {
      kr[u2] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, goff[u2], 0, 0));
      vr[u2] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, goff[u2], 0, 0));
    }
  };
  // this thread's first granule in a tile; granule u2 is GT / NG rows below
  // it, a constant the LDS writes take as their immediate offset
  static_assert(GT % NG == 0, "granule rows");
  const int st_k = (gtid / NG) * KST + (gtid % NG) * 8;
  const int st_v = (gtid / NG) * VST + (gtid % NG) * 8;
  auto stage = [&](int b) {
    _Float16* k_lds = tile_k(b) + st_k;
    _Float16* v_lds = tile_k(b) + TOK * KST + st_v;
#pragma unroll
    for (int u = 0; u < GPT; ++u) {
      *reinterpret_cast<u32x4*>(k_lds + u * (GT / NG) * KST) = kr[u];
      *reinterpret_cast<u32x4*>(v_lds + u * (GT / NG) * VST) = vr[u];
    }
  };
  auto compute = [&](int u, int b) {
    const _Float16* k_lds = tile_k(b);
    const _Float16* v_lds = k_lds + TOK * KST;
    int j, r0;
    unit_pos(u, j, r0);
    const int c0 = chunk_start(j) + r0;                     // position of the unit's first row
    const int len = min(TOK, chunk_end(j) - c0);            // rows of the unit
    if (len <= 0 || c0 > pos_last) return;                  // nothing the tile can see (uniform)

    // S^T for the unit's token slots: tile jt holds tokens 16jt..16jt+15;
    // each K read feeds the wavefront's QT query tiles. All of the unit's K
    // fragments are read first (one wait), then the JT independent
    // accumulation chains are interleaved on the matrix cores.
    floatx4 sacc[QT][JT];
    half8 ka[JT][KS];
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int s = 0; s < KS; ++s)
        ka[jt][s] = *reinterpret_cast<const half8*>(k_lds + (16 * jt + l16) * KST + 32 * s + 8 * g);
#pragma unroll
    for (int jt = 0; jt < JT; ++jt)
#pragma unroll
      for (int t = 0; t < QT; ++t) sacc[t][jt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int t = 0; t < QT; ++t)
          sacc[t][jt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ka[jt][s], qf[t][s], sacc[t][jt], 0, 0, 0);
    // lane holds S^T[token 16jt + 4g + i][row l16 of tile t] (unscaled).
    // Units that are whole and end before the tile's first position need no
    // mask (uniform test).
    if (len < TOK || c0 + TOK - 1 > pos_first) {
#pragma unroll
      for (int t = 0; t < QT; ++t)
#pragma unroll
        for (int jt = 0; jt < JT; ++jt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int tk = 16 * jt + 4 * g + i;
            if (!(tk < len && c0 + tk <= pos[t])) sacc[t][jt][i] = -INFINITY;
          }
    }
    half8 pb[QT][PV];
    bool moved = false;
    float alpha[QT];
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      float lmax = -INFINITY;
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int i = 0; i < 4; ++i) lmax = fmaxf(lmax, sacc[t][jt][i]);
      lmax = rows4_max(lmax);
      // Reference maximum in scaled base-2 units (qscale > 0 commutes with
      // max), moved only when the unit's maximum exceeds it by more than
      // kPfLazyMax: P = exp2(S - m) then stays <= 2^kPfLazyMax (fp16 keeps
      // its relative precision there) and the O accumulators are rescaled
      // in far fewer steps. Any reference gives the same O / n; partials
      // carry the one they used. (0.3 us less on a 512-token join.)
      const float lm = lmax * P.qscale;
      const float mn = lm > m_run[t] + kPfLazyMax ? lm : m_run[t];
      alpha[t] = fast_exp2(m_run[t] - mn);
      moved |= mn != m_run[t];
      m_run[t] = mn;
      half4 ph[JT];
#pragma unroll
      for (int jt = 0; jt < JT; ++jt) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          ph[jt][i] = static_cast<_Float16>(fast_exp2(__builtin_fmaf(sacc[t][jt][i], P.qscale, -mn)));
      }
      // O^T += V^T P^T over 32 tokens per 16x16x32 MFMA: lane group g's
      // 8-token K-slice is tokens 4g..4g+3 of token tiles 2p and 2p+1 (any
      // token order works as long as both operands share it), which is
      // exactly what the lane holds of P^T; two transposing reads fetch the
      // V^T side.
#pragma unroll
      for (int p2 = 0; p2 < PV; ++p2)
        pb[t][p2] = __builtin_shufflevector(ph[2 * p2], ph[2 * p2 + 1], 0, 1, 2, 3, 4, 5, 6, 7);
    }
    // O is rescaled only when some row's maximum moved (uniform test)
    if (__any(moved)) {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[t][dt] *= alpha[t];
        nacc[t] *= alpha[t];
      }
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int p2 = 0; p2 < PV; ++p2) {
        const _Float16* vp = v_lds + (32 * p2 + 4 * g + (l16 >> 2)) * VST + 16 * dt + 4 * (l16 & 3);
        const half4 v0 = lds_read_tr16(vp);             // tokens 32p + 4g + j
        const half4 v1 = lds_read_tr16(vp + 16 * VST);  // tokens 32p + 16 + 4g + j
        const half8 va = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int t = 0; t < QT; ++t)
          acc[t][dt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, pb[t][p2], acc[t][dt], 0, 0, 0);
      }
    }
    // n += the sum of P over the unit's tokens, from the same fp16 P as O:
    // an all-ones A operand makes every output row that sum (two matrix-core
    // ops instead of sixteen vector adds and a cross-lane reduction; with the
    // LDS writes' folded offsets, 0.27 us less on a 512-token join)
#pragma unroll
    for (int p2 = 0; p2 < PV; ++p2)
#pragma unroll
      for (int t = 0; t < QT; ++t)
        nacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones8, pb[t][p2], nacc[t], 0, 0, 0);
  };
  // Two LDS tiles per group: step i computes the group's unit i of the part
  // (unit u_lo + grp + i * NGRP) from tile i % 2 while unit i + 1 is written
  // into the other tile and unit i + 2 loads into the registers; one barrier
  // per step (after it, tile i % 2 is complete and nobody still reads the
  // other one).
  const int steps = (u_hi - u_lo + NGRP - 1) / NGRP;  // the same in every group
  if (steps > 0) {
    issue(u_lo + grp);
    stage(0);
    issue(u_lo + grp + NGRP);
  }
  for (int i = 0; i < steps; ++i) {
    __syncthreads();
    if (i + 1 < steps) {
      stage((i + 1) & 1);
      issue(u_lo + grp + (i + 2) * NGRP);
    }
    const int u = u_lo + grp + i * NGRP;
    if (u < u_hi) compute(u, i & 1);
  }
  // each lane's row sum (all four entries of nacc hold it)
  float n_row[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) n_row[t] = nacc[t][0];
  if constexpr (NGRP > 1) {
    // groups 1.. hand their (m, n, O) to group 0 through LDS (Eqn 2)
    float* ob = reinterpret_cast<float*>(lds);                    // [NGRP-1][64][OST]
    float* mb = ob + (NGRP - 1) * 64 * OST;                        // [NGRP-1][64][2]
    __syncthreads();  // the tiles are free
    if (grp > 0) {
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        const int r = 16 * (QT * w + t) + l16;
        float* o_ = ob + ((grp - 1) * 64 + r) * OST;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          *reinterpret_cast<floatx4*>(o_ + 16 * dt + 4 * g) = acc[t][dt];
        if (g == 0) {
          mb[((grp - 1) * 64 + r) * 2] = m_run[t];
          mb[((grp - 1) * 64 + r) * 2 + 1] = n_row[t];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      if (grp > 0) break;
      const int r = 16 * (QT * w + t) + l16;
#pragma unroll
      for (int k = 1; k < NGRP; ++k) {
        const float mo = mb[((k - 1) * 64 + r) * 2], no = mb[((k - 1) * 64 + r) * 2 + 1];
        const float M = fmaxf(m_run[t], mo);
        const float ws = fast_exp2(m_run[t] - M), wo = fast_exp2(mo - M);
        const float* o_ = ob + ((k - 1) * 64 + r) * OST;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
          acc[t][dt] = acc[t][dt] * ws + *reinterpret_cast<const floatx4*>(o_ + 16 * dt + 4 * g) * wo;
        n_row[t] = n_row[t] * ws + no * wo;
        m_run[t] = M;
      }
    }
  }
  if (S == 1) {
    if (grp > 0) return;
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      if (qi[t] < n_q) {
        const float inv = 1.f / n_row[t];
        _Float16* out = P.o + (static_cast<size_t>(qi[t]) * H + h) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          half4 r4;
#pragma unroll
          for (int i = 0; i < 4; ++i) r4[i] = static_cast<_Float16>(acc[t][dt][i] * inv);
          *reinterpret_cast<half4*>(out + 16 * dt + 4 * g) = r4;
        }
      }
    }
    return;
  }
  // A part of a split tile: group 0 publishes the block's (O, m, n) for the
  // tile's 64 rows (device-scope stores), the block counts its arrival, and
  // the last of the S parts folds all of them (Eqn 2: common maximum, each
  // part's sum and O rescaled) and writes o = O / n.
  constexpr int PF = kpf_part_floats<D>();
  constexpr int NT = 64 * WPG * NGRP;  // threads of the block
  const __amdgpu_buffer_rsrc_t rs = part_rsrc(P.ws, P.ws_bytes);
  if (grp == 0) {
    const uint32_t pw = static_cast<uint32_t>((static_cast<size_t>(tix) * S + part) * PF);
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int r = 16 * (QT * w + t) + l16;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        st_dev4(rs, 4 * (pw + r * D + 16 * dt + 4 * g), acc[t][dt][0], acc[t][dt][1], acc[t][dt][2],
                acc[t][dt][3]);
      if (g == 0) {
        st_dev(P.ws + pw + 64 * D + r, m_run[t]);
        st_dev(P.ws + pw + 64 * D + 64 + r, n_row[t]);
      }
    }
  }
  wait_stores();
  __syncthreads();  // every store of the block's part has completed
  __shared__ int last_part;
  if (tid == 0) last_part = arrive_last(P.cnt + tix, S);
  __syncthreads();
  if (!last_part) return;
  // The last part folds, online over batches of KB parts (Eqn 2 per output
  // item: running maximum, sum and O rescaled at each batch); each batch's
  // loads (O, m and n of every item's row in every part) are in flight
  // together.
  const size_t pt = static_cast<size_t>(tix) * S * PF;
  constexpr int IPT = 64 * (D / 4) / NT;  // 4-column items per thread
  constexpr int KB = 4;
  static_assert(IPT * NT == 64 * (D / 4), "fold items");
  float4 o4[IPT];
  float mx[IPT], nx[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    o4[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    mx[j] = kNegBig;
    nx[j] = 0.f;
  }
  for (int k0 = 0; k0 < S; k0 += KB) {
    float mk[KB][IPT], nk[KB][IPT];
    float4 vk[KB][IPT];
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      if (k0 + kk >= S) break;
      const size_t base = pt + static_cast<size_t>(k0 + kk) * PF;
#pragma unroll
      for (int j = 0; j < IPT; ++j) {
        const int e = tid + NT * j, r = e / (D / 4), d0 = 4 * (e % (D / 4));
        mk[kk][j] = ld_dev(P.ws + base + 64 * D + r);
        nk[kk][j] = ld_dev(P.ws + base + 64 * D + 64 + r);
        vk[kk][j] = ld_dev4(rs, static_cast<uint32_t>(4 * (base + r * D + d0)));
      }
    }
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      if (k0 + kk >= S) break;
#pragma unroll
      for (int j = 0; j < IPT; ++j) {
        const float M = fmaxf(mx[j], mk[kk][j]);
        const float a = fast_exp2(mx[j] - M), b = fast_exp2(mk[kk][j] - M);
        o4[j].x = o4[j].x * a + vk[kk][j].x * b;
        o4[j].y = o4[j].y * a + vk[kk][j].y * b;
        o4[j].z = o4[j].z * a + vk[kk][j].z * b;
        o4[j].w = o4[j].w * a + vk[kk][j].w * b;
        nx[j] = nx[j] * a + nk[kk][j] * b;
        mx[j] = M;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int e = tid + NT * j, r = e / (D / 4), d0 = 4 * (e % (D / 4));
    if (q0 + r >= n_q) continue;
    const float f = 1.f / nx[j];
    half4 r4;
    r4[0] = static_cast<_Float16>(o4[j].x * f);
    r4[1] = static_cast<_Float16>(o4[j].y * f);
    r4[2] = static_cast<_Float16>(o4[j].z * f);
    r4[3] = static_cast<_Float16>(o4[j].w * f);
    *reinterpret_cast<half4*>(P.o + (static_cast<size_t>(q0 + r) * H + h) * D + d0) = r4;
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, hipStream_t stream) {
  if (a.n_q <= 0 || a.n_chunks <= 0) return hipSuccess;
  KpfParams P{static_cast<const _Float16*>(a.q), static_cast<_Float16*>(a.o),
              static_cast<const _Float16*>(a.kpool), static_cast<const _Float16*>(a.vpool), a.ss,
              a.hs, a.n_chunks, a.n_q, a.H, a.C, a.qscale, a.n_split, a.ws, a.cnt,
              static_cast<uint32_t>(a.ws_bytes)};
  if (a.n_split < 1 || (a.n_split > 1 && (!a.ws || !a.cnt || a.ws_bytes > 0xFFFFFFF0ull)))
    return hipErrorInvalidValue;
  // two groups of four wavefronts (16 queries each), 64-row units, two LDS
  // tiles per group
  constexpr int kGroups = 2, kWaves = 4, kTok = 64;
  // paths up to this long keep their chunk table in the lanes of a register
  constexpr int kLaneChunks = 64;
  const int blocks = ((a.n_q + 63) / 64) * a.H * a.n_split;
  const dim3 grid(8 * ((blocks + 7) / 8));  // a multiple of the XCD count
  const dim3 block(64 * kWaves * kGroups);
  if (a.host_path && a.n_chunks <= kLaneChunks) {
    KpfPath<kLaneChunks> path;
    for (int j = 0; j < a.n_chunks; ++j) path.slot[j] = a.host_path[j];
    for (int j = 0; j <= a.n_chunks; ++j) path.start[j] = a.host_path[a.n_chunks + j];
    if (a.D == 128)
      kpf_kernel<128, kGroups, kWaves, kTok, kLaneChunks><<<grid, block, 0, stream>>>(
          P, nullptr, nullptr, path);
    else if (a.D == 64)
      kpf_kernel<64, kGroups, kWaves, kTok, kLaneChunks><<<grid, block, 0, stream>>>(
          P, nullptr, nullptr, path);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (a.host_path && a.n_chunks <= kPrefillInlineChunks) {
    KpfPath<kPrefillInlineChunks> path;
    for (int j = 0; j < a.n_chunks; ++j) path.slot[j] = a.host_path[j];
    for (int j = 0; j <= a.n_chunks; ++j) path.start[j] = a.host_path[a.n_chunks + j];
    if (a.D == 128)
      kpf_kernel<128, kGroups, kWaves, kTok, kPrefillInlineChunks><<<grid, block, 0, stream>>>(
          P, nullptr, nullptr, path);
    else if (a.D == 64)
      kpf_kernel<64, kGroups, kWaves, kTok, kPrefillInlineChunks><<<grid, block, 0, stream>>>(
          P, nullptr, nullptr, path);
    else return hipErrorInvalidValue;
    return hipGetLastError();
  }
  if (!a.chunk_slot) return hipErrorInvalidValue;
  const KpfPath<1> none{};
  if (a.D == 128)
    kpf_kernel<128, kGroups, kWaves, kTok, 0><<<grid, block, 0, stream>>>(P, a.chunk_slot,
                                                                         a.chunk_start, none);
  else if (a.D == 64)
    kpf_kernel<64, kGroups, kWaves, kTok, 0><<<grid, block, 0, stream>>>(P, a.chunk_slot,
                                                                        a.chunk_start, none);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace ca
