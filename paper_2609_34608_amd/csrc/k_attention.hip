// Bidirectional softmax attention over the joint token sequence (gfx950).
//
// qkv_relayout: [B*T][3D] projection output -> per-head q, k ([B*H][Tpad][dh],
// RMS-normalised with gains when QK-norm is on) and v transposed
// ([B*H][dh][Tpad]).  Pad rows/columns beyond T are never written; the host
// zero-fills them once.
//
// bf16 flash attention (dh = 64): each wave owns 16*QT queries and keeps their
// Q fragments in registers.  Scores are formed transposed, S^T = K Q^T, with
// v_mfma_f32_16x16x32_bf16 so that a lane's accumulators all belong to one
// query column: the online-softmax rescale of O^T = V^T P^T is lane-local and
// the running max needs only two cross-lane steps.  P^T feeds the second MFMA
// straight from registers; the key order inside the 32-key contraction is the
// one the score accumulators hold, and the QKV epilogue stores V^T with its
// keys permuted to match (vt_key_pos), so each V^T operand is one 16-byte LDS
// read.  K and V^T tiles of 64 keys (128-byte rows, 16-byte chunks XOR-swizzled
// by row & 7: conflict-free ds_read_b128) go through ST LDS stages filled by
// global_load_lds_dwordx4, ST-1 in flight.  Softmax runs in fp32 with exp2: q
// arrives pre-scaled by log2(e)/sqrt(dh) (QKV epilogue), and the score
// accumulators start at -m, the query's running max, so a score comes out of
// the MFMA as its exp2 argument.  m only moves (and O is only rescaled) when
// a tile raises a query's max by more than 8, which keeps every p <= 2^8 and
// leaves the normalised result unchanged; the first tile always sets it.  The
// softmax denominator is one more MFMA per 32 keys (a ones operand against
// P^T), summing exactly the bf16 P that multiplies V.
#include <math.h>

#include "wam_internal.h"

namespace wam {

namespace {

// ------------------------------------------------------------- relayout
template <typename T, int DH>
__global__ __launch_bounds__(256) void qkv_relayout_kernel(RelayoutArgs a) {
  if (a.skip && *a.skip) return;
  constexpr int TT = 64;  // tokens per block
  __shared__ float vs[DH][TT + 1];
  const int t0 = blockIdx.x * TT, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid % kWave, wid = tid / kWave;
  const T* qkv = static_cast<const T*>(a.qkv);
  const size_t bh = (size_t)b * a.H + h;
  T* qo = static_cast<T*>(a.q) + bh * a.Tpad * DH;
  T* ko = static_cast<T*>(a.k) + bh * a.Tpad * DH;
  T* vo = static_cast<T*>(a.vt) + bh * DH * a.Tpad;
  // q and k: one wave per token row, lane = feature (DH <= 64)
  for (int tt = wid; tt < TT; tt += 4) {
    const int t = t0 + tt;
    if (t >= a.T) break;
    const T* src = qkv + ((size_t)b * a.T + t) * 3 * a.D + h * DH;
    float qv = lane < DH ? to_f32(src[lane]) : 0.f;
    float kv = lane < DH ? to_f32(src[a.D + lane]) : 0.f;
    const float vv = lane < DH ? to_f32(src[2 * a.D + lane]) : 0.f;
    if (a.qk_norm) {
      const float rq = rsqrtf(wave_sum(qv * qv) / (float)DH + a.eps);
      const float rk = rsqrtf(wave_sum(kv * kv) / (float)DH + a.eps);
      if (lane < DH) {
        qv = qv * rq * a.q_g[lane];
        kv = kv * rk * a.k_g[lane];
      }
    }
    if (lane < DH) {
      qo[(size_t)t * DH + lane] = from_f32<T>(qv);
      ko[(size_t)t * DH + lane] = from_f32<T>(kv);
      vs[lane][tt] = vv;
    }
  }
  __syncthreads();
  // v^T: row d holds tokens t0 .. t0+63 contiguously
  for (int i = tid; i < DH * TT; i += 256) {
    const int d = i / TT, tt = i % TT;
    const int t = t0 + tt;
    if (t < a.T) vo[(size_t)d * a.Tpad + t] = from_f32<T>(vs[d][tt]);
  }
}

// ------------------------------------------------------------- bf16 flash attention
constexpr int kDh = 64;
constexpr int kKB = 64;  // keys per tile
// largest fixed softmax reference: p >= 2^(-2 mref) must stay a normal float
constexpr float kMaxBoundedRef = 60.0f;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void global_void;

// Query block and (sample, head) of this workgroup.  Workgroups go to the 8
// XCDs round-robin by linear id; renumbering them so that each XCD takes a
// contiguous run of (head, query block) pairs keeps all query blocks of a
// head on one XCD, whose L2 then fetches that head's K and V^T once.
__device__ __forceinline__ void attn_block(int& qb, int& bh) {
  const int nqb = gridDim.x, nb = gridDim.x * gridDim.y;
  const int lin = blockIdx.y * nqb + blockIdx.x;
  const int per = nb / 8, rem = nb % 8, x = lin % 8, idx = lin / 8;
  const int logical = x * per + min(x, rem) + idx;
  qb = logical % nqb;
  bh = logical / nqb;
}

// s_waitcnt immediate (gfx9 layout): at most n vector-memory operations and no
// LDS operation outstanding
constexpr int waitcnt_vm_lgkm0(int n) { return (n & 0xf) | ((n >> 4) << 14) | (0x7 << 4); }
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// BND: the fixed reference of the bounded kernels (a.mref) instead of the
// running max, in this plain (not software-pipelined) loop, which needs one
// score buffer and so leaves room for more waves per SIMD.
// KSPLIT > 1 (bounded only): KSPLIT groups of NW waves take the same queries
// and split the keys, group g taking key tiles g, g + KSPLIT, ...  With a
// fixed reference the partial O and l of the groups simply add (no
// rescaling), which group 0 does at the end through LDS, in group order.
// This shortens the serial chain of key tiles per wave where the grid is too
// small to fill the chip (short sequences).
template <int QT, int NW, int ST, bool BND = false, int KSPLIT = 1>
__global__ __launch_bounds__(NW * KSPLIT * 64) void attn_bf16_kernel(AttnArgs a) {
  constexpr int QB = NW * QT * 16;  // queries per block
  constexpr int NWT = NW * KSPLIT;  // waves per block
  // 1 KiB load instructions per stage: per key tile K rows 0-63, V^T rows 64-127
  constexpr int NI = 16 * KSPLIT;
  constexpr int IPW = NI / NWT;
  static_assert(IPW >= 1 && IPW * NWT == NI, "stage load split");
  static_assert(ST >= 2 && (ST - 2) * IPW < 64, "stage count");
  static_assert(KSPLIT == 1 || BND, "key split needs the fixed reference");
  if (a.skip && *a.skip) return;
  // stage: KSPLIT key tiles of 128 rows of 64 bf16 (128 bytes); chunk c of
  // row r stored at c ^ (r & 7)
  __shared__ __attribute__((aligned(1024))) bf16 sm[ST][KSPLIT * 128 * kDh];

  int qb, bh;
  attn_block(qb, bh);
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, lane = tid % 64, wid = tid / 64;
  const int kgrp = wid / NW, wl = wid % NW;
  const int q0 = qb * QB + wl * QT * 16;
  const int g = lane / 16, lr = lane % 16;

  const bf16* Q = static_cast<const bf16*>(a.q) + (size_t)bh * a.Tpad * kDh;
  const bf16* Kg = static_cast<const bf16*>(a.k) + (size_t)bh * a.Tpad * kDh;
  const bf16* Vg = static_cast<const bf16*>(a.vt) + (size_t)bh * kDh * a.Tpad;

  // Q fragments (B operand of S^T = K Q^T): query q0 + qt*16 + lr, dh chunk c
  bf16x8 qf[QT][2];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int q = q0 + qt * 16 + lr;
      qf[qt][c] = q < a.Tpad ? *reinterpret_cast<const bf16x8*>(Q + (size_t)q * kDh + c * 32 + g * 8)
                             : bf16x8{};
    }

  f32x4 o[4][QT];  // O^T tiles: dh tile x query tile
  f32x4 l[QT];     // softmax denominators (all four elements equal)
  float mrun[QT];  // running max, log2 units; 0 until the first tile sets it
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
    for (int d = 0; d < 4; ++d) o[d][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    l[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    mrun[qt] = 0.f;
  }
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = static_cast<bf16>(1.0f);

  // Load instruction j of this wave fills stage rows 8*i .. 8*i+7 with
  // i = wid + NWT*j; lane l writes chunk l%8 of row l/8, i.e. global chunk
  // (l%8) ^ (row & 7).  Stage rows 128u .. 128u+127 hold key tile u of the
  // stage's KSPLIT tiles: rows 0-63 are keys (K rows), rows 64-127 are dh
  // rows of V^T; the next key tile is 64 K rows or 64 V^T columns further on.
  const bf16* src[IPW];
  int sub[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int i = wid + NWT * j;
    const int row = 8 * (i % 16) + lane / 8;
    const int col = ((lane % 8) ^ (row & 7)) * 8;
    sub[j] = i / 16;
    src[j] = row < 64 ? Kg + (size_t)row * kDh + col : Vg + (size_t)(row - 64) * a.Tpad + col;
  }
  const int nkb = a.Tpad / kKB;
  // stage kp holds key tiles KSPLIT kp + u (past the last tile: the last tile
  // again, into rows nobody reads)
  auto issue = [&](auto S, int kp) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int i = wid + NWT * j;
      // one tile per stage: instructions j < IPW/2 carry K rows for every wave
      const bool krow = KSPLIT == 1 ? j < IPW / 2 : (i % 16) < 8;
      const int kb = KSPLIT == 1 ? kp : min(kp * KSPLIT + sub[j], nkb - 1);
      const size_t step = krow ? (size_t)kKB * kDh : (size_t)kKB;
      __builtin_amdgcn_global_load_lds((const global_void*)(src[j] + kb * step),
                                       (lds_void*)(&sm[s][i * 512]), 16, 0, 0);
    }
  };

  const int sw = lr & 7;  // swizzle of every row this lane reads (tile rows are multiples of 16)
  auto block = [&](auto S, int k0, auto MASK, bool first) __attribute__((always_inline)) {
    const bf16* st = sm[decltype(S)::value] + (KSPLIT > 1 ? kgrp * 128 * kDh : 0);
    // S^T - m tiles [key tile kt][query tile qt]: the accumulators start at -m
    f32x4 s[4][QT];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const bf16* krow = st + (kt * 16 + lr) * kDh;
      const bf16x8 k0f = *reinterpret_cast<const bf16x8*>(krow + ((g ^ sw) * 8));
      const bf16x8 k1f = *reinterpret_cast<const bf16x8*>(krow + (((g + 4) ^ sw) * 8));
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const float nm = BND ? -a.mref : -mrun[qt];
        f32x4 z = {nm, nm, nm, nm};
        z = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0f, qf[qt][0], z, 0, 0, 0);
        s[kt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1f, qf[qt][1], z, 0, 0, 0);
      }
    }
    // mask keys >= T (key of element r: k0 + kt*16 + 4g + r); only the last
    // key tile can hold such keys, so only its instance carries the mask
    if constexpr (decltype(MASK)::value) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool live = k0 + kt * 16 + g * 4 + r < a.T;
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) s[kt][qt][r] = live ? s[kt][qt][r] : -INFINITY;
        }
    }
    if constexpr (!BND) {
    // online softmax per query column (lane-local except the max)
    float mx[QT];
    bool grow = false;
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float m = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) m = fmaxf(m, s[kt][qt][r]);
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      mx[qt] = m;
      grow = grow || m > 8.0f;
    }
    // move m when this tile raises some query's max by more than 8 (one
    // wave-uniform branch for all query tiles), and always on the first tile
    if (first || __builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const float delta = first ? mx[qt] : fmaxf(mx[qt], 0.f);
        // first tile: O and l are still zero, any finite factor keeps them so
        const float corr = __builtin_amdgcn_exp2f(fminf(-delta, 0.f));
        mrun[qt] += delta;
        l[qt] *= corr;
#pragma unroll
        for (int d = 0; d < 4; ++d) o[d][qt] *= corr;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) s[kt][qt] -= delta;
      }
    }
    }
    // V^T operands: with the stored key order the eight keys of slot (c, g)
    // are chunk 4c + g of the V^T row
    bf16x8 vf[4][2];
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        vf[d][c] = *reinterpret_cast<const bf16x8*>(st + (64 + d * 16 + lr) * kDh + (((4 * c + g) ^ sw) * 8));
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      // B operand of O^T += V^T P^T for key chunk c: slots 0-3 = key tile 2c,
      // slots 4-7 = key tile 2c+1 (keys 4g+r within each)
      bf16x8 pf[2];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pf[c][r] = static_cast<bf16>(__builtin_amdgcn_exp2f(s[2 * c][qt][r]));
          pf[c][4 + r] = static_cast<bf16>(__builtin_amdgcn_exp2f(s[2 * c + 1][qt][r]));
        }
      }
      // the ones operand adds the column sums of P^T into l
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        l[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[c], l[qt], 0, 0, 0);
#pragma unroll
        for (int d = 0; d < 4; ++d) o[d][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[d][c], pf[c], o[d][qt], 0, 0, 0);
      }
    }
  };

  // one stage (KSPLIT key tiles) on slot J: this wave's loads of stage kp
  // have landed and its LDS reads are done; after the barrier everyone's are,
  // and the slot of the previous stage takes stage kp+ST-1 (past the end the
  // last stage again, into slots nobody reads, which keeps the wait counts
  // uniform).  Group kgrp works on key tile KSPLIT kp + kgrp.
  const int nkp = (nkb + KSPLIT - 1) / KSPLIT;
  const bool live = q0 < a.T;
  const std::integral_constant<bool, false> nomask{};
  const std::integral_constant<bool, true> withmask{};
  auto step = [&](auto J, int kp, auto TAIL) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 2) * IPW));
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(std::integral_constant<int, (j + ST - 1) % ST>{}, min(kp + ST - 1, nkp - 1));
    __builtin_amdgcn_sched_barrier(0);  // loads leave before the MFMAs, not sunk below them
    const int kb = kp * KSPLIT + kgrp;
    // a wave whose queries all lie past T (the last query block of a head)
    // still loads and synchronises but computes nothing
    if (!live) return;
    if constexpr (!decltype(TAIL)::value) {
      block(J, kb * kKB, nomask, kb == 0);
    } else {
      // the last stage: the last key tile carries the padded keys, and with
      // a key split some group may have no tile left
      if (kb < nkb - 1) block(J, kb * kKB, nomask, kb == 0);
      else if (kb == nkb - 1) block(J, kb * kKB, withmask, kb == 0);
    }
  };
  static_for<ST - 1>([&](auto P) __attribute__((always_inline)) { issue(P, min((int)decltype(P)::value, nkp - 1)); });
  // stages 0 .. nkp-2 carry no padded keys; the last one runs as the tail
  const int nbody = nkp - 1;
  const int nfull = nbody / ST * ST;
  for (int kp0 = 0; kp0 < nfull; kp0 += ST)
    static_for<ST>([&](auto J) __attribute__((always_inline)) { step(J, kp0 + decltype(J)::value, nomask); });
  static_for<ST>([&](auto J) __attribute__((always_inline)) {
    const int kp = nfull + decltype(J)::value;
    if (kp < nbody) step(J, kp, nomask);
    else if (kp == nbody) step(J, kp, withmask);
  });
  // no load may still be writing this block's LDS when the block retires
  __builtin_amdgcn_s_waitcnt(0);

  if constexpr (KSPLIT > 1) {
    // groups 1.. hand O and l to group 0 through the idle stages
    static_assert((KSPLIT - 1) * NW * 5 * QT * 64 * 16 <= ST * KSPLIT * 128 * kDh * 2, "LDS for the key-split sum");
    f32x4* xch = reinterpret_cast<f32x4*>(&sm[0][0]);
    __syncthreads();
    if (kgrp > 0) {
      f32x4* w = xch + ((kgrp - 1) * NW + wl) * 5 * QT * 64 + lane;
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
        for (int d = 0; d < 4; ++d) w[(qt * 5 + d) * 64] = o[d][qt];
        w[(qt * 5 + 4) * 64] = l[qt];
      }
    }
    __syncthreads();
    if (kgrp > 0) return;
#pragma unroll
    for (int g2 = 1; g2 < KSPLIT; ++g2) {
      const f32x4* w = xch + ((g2 - 1) * NW + wl) * 5 * QT * 64 + lane;
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
        for (int d = 0; d < 4; ++d) o[d][qt] += w[(qt * 5 + d) * 64];
        l[qt] += w[(qt * 5 + 4) * 64];
      }
    }
  }

  // normalise and store O[b*T + q][h*64 + dh]; lane holds dh = d*16 + 4g + r of query lr
  bf16* out = static_cast<bf16*>(a.out);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float inv = 1.0f / l[qt][0];
    const int q = q0 + qt * 16 + lr;
    if (q >= a.T) continue;
    bf16* orow = out + ((size_t)b * a.T + q) * a.D + h * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      bf16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = static_cast<bf16>(o[d][qt][r] * inv);
      *reinterpret_cast<bf16x4*>(orow + d * 16 + g * 4) = v;
    }
  }
}

// ------------------------------------------------------------- bf16 attention, bounded scores
// When every score of the layer is known to lie in [-mref, mref] (QK-norm on:
// |q.k| <= |q| |k| is fixed by the head size and the gains), the softmax
// reference is the constant mref instead of a running max: softmax does not
// depend on the reference, p = 2^(s - mref) stays in [2^-2mref, 1], and the
// loop carries no max, no cross-lane step and no rescale.  The loop is also
// software-pipelined: the S^T MFMAs of key tile j+1 are issued before the
// exp2 of tile j, so the matrix cores work on the next tile while the VALU
// turns the current one into P.  Stage slots: tile t sits in slot t % ST;
// iteration j reads tiles j (V^T) and j+1 (K) and refills the slot of tile
// j-1, so ST >= 3 and ST-3 tiles stay in flight across the barrier.
template <int QT, int NW, int ST>
__global__ __launch_bounds__(NW * 64) void attn_bf16_bounded_kernel(AttnArgs a) {
  constexpr int QB = NW * QT * 16;
  constexpr int NI = 16;
  constexpr int IPW = NI / NW;
  constexpr int U = ST % 2 == 0 ? ST : 2 * ST;  // unroll: slot and S buffer indices both static
  static_assert(IPW >= 1 && IPW * NW == NI, "stage load split");
  static_assert(ST >= 3 && (ST - 2) * IPW < 64, "stage count");
  if (a.skip && *a.skip) return;
  __shared__ __attribute__((aligned(1024))) bf16 sm[ST][128 * kDh];

  int qb, bh;
  attn_block(qb, bh);
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, lane = tid % 64, wid = tid / 64;
  const int q0 = qb * QB + wid * QT * 16;
  const int g = lane / 16, lr = lane % 16;

  const bf16* Q = static_cast<const bf16*>(a.q) + (size_t)bh * a.Tpad * kDh;
  const bf16* Kg = static_cast<const bf16*>(a.k) + (size_t)bh * a.Tpad * kDh;
  const bf16* Vg = static_cast<const bf16*>(a.vt) + (size_t)bh * kDh * a.Tpad;

  bf16x8 qf[QT][2];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int q = q0 + qt * 16 + lr;
      qf[qt][c] = q < a.Tpad ? *reinterpret_cast<const bf16x8*>(Q + (size_t)q * kDh + c * 32 + g * 8)
                             : bf16x8{};
    }

  f32x4 o[4][QT];
  f32x4 l[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
    for (int d = 0; d < 4; ++d) o[d][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    l[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = static_cast<bf16>(1.0f);
  const float nm = -a.mref;

  // load instruction j of this wave: stage rows 8*(wid + NW*j) .. +7, as in
  // the running-max kernel
  const bf16* src[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int row = 8 * (wid + NW * j) + lane / 8;
    const int col = ((lane % 8) ^ (row & 7)) * 8;
    src[j] = j < IPW / 2 ? Kg + (size_t)row * kDh + col : Vg + (size_t)(row - 64) * a.Tpad + col;
  }
  auto issue = [&](auto S, int kb) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const size_t step = j < IPW / 2 ? (size_t)kKB * kDh : (size_t)kKB;
      __builtin_amdgcn_global_load_lds((const global_void*)(src[j] + kb * step),
                                       (lds_void*)(&sm[s][(wid + NW * j) * 512]), 16, 0, 0);
    }
  };

  const int sw = lr & 7;
  f32x4 sc[2][4][QT];  // S^T - mref of two key tiles: tile t in sc[t % 2]
  auto qk = [&](auto S, auto BUF) __attribute__((always_inline)) {
    const bf16* st = sm[decltype(S)::value];
    constexpr int bi = decltype(BUF)::value;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const bf16* krow = st + (kt * 16 + lr) * kDh;
      const bf16x8 k0f = *reinterpret_cast<const bf16x8*>(krow + ((g ^ sw) * 8));
      const bf16x8 k1f = *reinterpret_cast<const bf16x8*>(krow + (((g + 4) ^ sw) * 8));
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        f32x4 z = {nm, nm, nm, nm};
        z = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0f, qf[qt][0], z, 0, 0, 0);
        sc[bi][kt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1f, qf[qt][1], z, 0, 0, 0);
      }
    }
  };
  auto pv = [&](auto S, auto BUF, int k0, auto MASK) __attribute__((always_inline)) {
    const bf16* st = sm[decltype(S)::value];
    constexpr int bi = decltype(BUF)::value;
    if constexpr (decltype(MASK)::value) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool live = k0 + kt * 16 + g * 4 + r < a.T;
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) sc[bi][kt][qt][r] = live ? sc[bi][kt][qt][r] : -INFINITY;
        }
    }
    bf16x8 vf[4][2];
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        vf[d][c] = *reinterpret_cast<const bf16x8*>(st + (64 + d * 16 + lr) * kDh + (((4 * c + g) ^ sw) * 8));
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      bf16x8 pf[2];
#pragma unroll
      for (int c = 0; c < 2; ++c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pf[c][r] = static_cast<bf16>(__builtin_amdgcn_exp2f(sc[bi][2 * c][qt][r]));
          pf[c][4 + r] = static_cast<bf16>(__builtin_amdgcn_exp2f(sc[bi][2 * c + 1][qt][r]));
        }
      }
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        l[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[c], l[qt], 0, 0, 0);
#pragma unroll
        for (int d = 0; d < 4; ++d) o[d][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[d][c], pf[c], o[d][qt], 0, 0, 0);
      }
    }
  };

  const int nkb = a.Tpad / kKB;
  const std::integral_constant<bool, false> nomask{};
  const std::integral_constant<bool, true> withmask{};
  // prologue: tiles 0 .. ST-2 in flight, wait for tile 0, S of tile 0
  static_for<ST - 1>([&](auto P) __attribute__((always_inline)) { issue(P, min((int)decltype(P)::value, nkb - 1)); });
  __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 2) * IPW));
  compiler_fence();
  __builtin_amdgcn_s_barrier();
  compiler_fence();
  qk(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});

  // iteration kb < nkb-1: tile kb+1 has landed everywhere and tile kb-1's slot
  // is free after the barrier; S of tile kb+1, then P and O of tile kb.  Past
  // the end the refill repeats the last tile into dead slots (uniform counts).
  auto body = [&](auto J, int kb) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 3) * IPW));
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    issue(std::integral_constant<int, (j + ST - 1) % ST>{}, min(kb + ST - 1, nkb - 1));
    __builtin_amdgcn_sched_barrier(0);  // loads leave before the MFMAs, not sunk below them
    qk(std::integral_constant<int, (j + 1) % ST>{}, std::integral_constant<int, (j + 1) % 2>{});
    pv(std::integral_constant<int, j % ST>{}, std::integral_constant<int, j % 2>{}, kb * kKB, nomask);
  };
  // the last tile: its S and its V^T stage are already resident
  auto last = [&](auto J, int kb) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    pv(std::integral_constant<int, j % ST>{}, std::integral_constant<int, j % 2>{}, kb * kKB, withmask);
  };
  const int nbody = nkb - 1;
  int kb0 = 0;
  for (; kb0 + U <= nbody; kb0 += U)
    static_for<U>([&](auto J) __attribute__((always_inline)) { body(J, kb0 + decltype(J)::value); });
  static_for<U>([&](auto J) __attribute__((always_inline)) {
    const int kb = kb0 + decltype(J)::value;
    if (kb < nbody) body(J, kb);
    else if (kb == nbody) last(J, kb);
  });
  __builtin_amdgcn_s_waitcnt(0);

  bf16* out = static_cast<bf16*>(a.out);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float inv = 1.0f / l[qt][0];
    const int q = q0 + qt * 16 + lr;
    if (q >= a.T) continue;
    bf16* orow = out + ((size_t)b * a.T + q) * a.D + h * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      bf16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = static_cast<bf16>(o[d][qt][r] * inv);
      *reinterpret_cast<bf16x4*>(orow + d * 16 + g * 4) = v;
    }
  }
}

// ------------------------------------------------------------- bf16 attention, bounded scores, ping-pong
// Same fixed-reference softmax as above, with the work of a key tile split
// into a matrix phase M(t) (S^T of tile t, then O += V^T P^T of tile t-1)
// and a vector phase V(t) (P of tile t = exp2 of S, packed to bf16).  The 8
// waves form two groups that share the block's K / V^T stages and run half a
// phase apart: waves w and w+4 sit on the same SIMD, and while one runs its
// MFMAs the other runs its exp2s, so the two pipes overlap instead of taking
// turns inside one wave.  Every phase ends at a block barrier: with intervals
// counted from 0, group 0 runs M(t) in interval 2t and V(t) in 2t+1, group 1
// runs M(t) in 2t+1 and V(t) in 2t+2.  Tile t is read in intervals 2t .. 2t+3
// (its K by both groups' M(t), its V^T by both groups' M(t+1)); the barrier
// that opens interval 2m checks that tile m has landed and refills the slot
// of tile m-2 with tile m+ST-2.
template <int QT, int ST>
__global__ __launch_bounds__(512) void attn_bf16_pingpong_kernel(AttnArgs a) {
  constexpr int NW = 8;
  constexpr int QB = NW * QT * 16;
  constexpr int NI = 16;
  constexpr int IPW = NI / NW;
  static_assert(ST >= 4 && (ST - 1) * IPW < 64, "stage count");
  if (a.skip && *a.skip) return;
  __shared__ __attribute__((aligned(1024))) bf16 sm[ST][128 * kDh];

  int qb, bh;
  attn_block(qb, bh);
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, lane = tid % 64, wid = tid / 64;
  const bool grp1 = wid >= 4;
  const int q0 = qb * QB + wid * QT * 16;
  const int g = lane / 16, lr = lane % 16;

  const bf16* Q = static_cast<const bf16*>(a.q) + (size_t)bh * a.Tpad * kDh;
  const bf16* Kg = static_cast<const bf16*>(a.k) + (size_t)bh * a.Tpad * kDh;
  const bf16* Vg = static_cast<const bf16*>(a.vt) + (size_t)bh * kDh * a.Tpad;

  bf16x8 qf[QT][2];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int q = q0 + qt * 16 + lr;
      qf[qt][c] = q < a.Tpad ? *reinterpret_cast<const bf16x8*>(Q + (size_t)q * kDh + c * 32 + g * 8)
                             : bf16x8{};
    }
  f32x4 o[4][QT];
  f32x4 l[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
#pragma unroll
    for (int d = 0; d < 4; ++d) o[d][qt] = f32x4{0.f, 0.f, 0.f, 0.f};
    l[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = static_cast<bf16>(1.0f);
  const float nm = -a.mref;

  const bf16* src[IPW];
#pragma unroll
  for (int j = 0; j < IPW; ++j) {
    const int row = 8 * (wid + NW * j) + lane / 8;
    const int col = ((lane % 8) ^ (row & 7)) * 8;
    src[j] = j < IPW / 2 ? Kg + (size_t)row * kDh + col : Vg + (size_t)(row - 64) * a.Tpad + col;
  }
  const int nkb = a.Tpad / kKB;
  auto issue = [&](int t) __attribute__((always_inline)) {
    const int slot = t % ST, kb = min(t, nkb - 1);
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const size_t step = j < IPW / 2 ? (size_t)kKB * kDh : (size_t)kKB;
      __builtin_amdgcn_global_load_lds((const global_void*)(src[j] + kb * step),
                                       (lds_void*)(&sm[slot][(wid + NW * j) * 512]), 16, 0, 0);
    }
  };
  // Barriers.  The scheduling barriers keep each phase's instructions between
  // its two block barriers (the compiler would otherwise merge the phases).
  // Barrier opening interval 2m: tile m has landed (every wave's part of it),
  // then the slot of tile m-2 takes tile m+ST-2 (at m = 1 that reloads tile
  // ST-1 into its own unread slot; tiles past the end repeat the last one
  // into dead slots), which keeps the wait counts uniform and the loop free
  // of branches.
  auto sync_even = [&](int m) __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 3) * IPW));
    compiler_fence();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compiler_fence();
    issue(m + ST - 2);
    __builtin_amdgcn_sched_barrier(0);  // loads leave before the phase's MFMAs
  };
  auto sync_odd = [&]() __attribute__((always_inline)) {
    compiler_fence();
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    compiler_fence();
  };

  const int sw = lr & 7;
  f32x4 sc[4][QT];
  bf16x8 pf[QT][2];
  // M(t): S^T of tile t (QK) and O += V^T P^T of tile t-1 (PV)
  auto mphase = [&](int t, auto QK, auto PV) __attribute__((always_inline)) {
    if constexpr (decltype(QK)::value) {
      const bf16* st = sm[t % ST];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const bf16* krow = st + (kt * 16 + lr) * kDh;
        const bf16x8 k0f = *reinterpret_cast<const bf16x8*>(krow + ((g ^ sw) * 8));
        const bf16x8 k1f = *reinterpret_cast<const bf16x8*>(krow + (((g + 4) ^ sw) * 8));
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          f32x4 z = {nm, nm, nm, nm};
          z = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0f, qf[qt][0], z, 0, 0, 0);
          sc[kt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1f, qf[qt][1], z, 0, 0, 0);
        }
      }
    }
    if constexpr (decltype(PV)::value) {
      const bf16* st = sm[(t - 1) % ST];
      bf16x8 vf[4][2];
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int c = 0; c < 2; ++c)
          vf[d][c] = *reinterpret_cast<const bf16x8*>(st + (64 + d * 16 + lr) * kDh + (((4 * c + g) ^ sw) * 8));
#pragma unroll
      for (int qt = 0; qt < QT; ++qt)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          l[qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[qt][c], l[qt], 0, 0, 0);
#pragma unroll
          for (int d = 0; d < 4; ++d)
            o[d][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[d][c], pf[qt][c], o[d][qt], 0, 0, 0);
        }
    }
  };
  // V(t): P of tile t; the last tile masks keys >= T
  auto vphase = [&](int t, auto MASK) __attribute__((always_inline)) {
    if constexpr (decltype(MASK)::value) {
      const int k0 = t * kKB;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool live = k0 + kt * 16 + g * 4 + r < a.T;
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) sc[kt][qt][r] = live ? sc[kt][qt][r] : -INFINITY;
        }
    }
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pf[qt][c][r] = static_cast<bf16>(__builtin_amdgcn_exp2f(sc[2 * c][qt][r]));
          pf[qt][c][4 + r] = static_cast<bf16>(__builtin_amdgcn_exp2f(sc[2 * c + 1][qt][r]));
        }
  };
  const std::integral_constant<bool, false> no{};
  const std::integral_constant<bool, true> yes{};

  static_for<ST>([&](auto P) __attribute__((always_inline)) { issue(decltype(P)::value); });
  __builtin_amdgcn_s_waitcnt(waitcnt_vm_lgkm0((ST - 1) * IPW));
  sync_odd();  // opens interval 0: tile 0 has landed everywhere
  // one straight-line program per group (no branch between the barriers)
  if (!grp1) {
    mphase(0, yes, no);
    sync_odd();
    for (int t = 1; t < nkb; ++t) {
      vphase(t - 1, no);
      sync_even(t);
      mphase(t, yes, yes);
      sync_odd();
    }
    vphase(nkb - 1, yes);
    sync_even(nkb);
    mphase(nkb, no, yes);
    sync_odd();  // both groups pass the same number of barriers
  } else {
    sync_odd();  // group 1 starts one interval later
    mphase(0, yes, no);
    sync_even(1);
    for (int t = 1; t < nkb; ++t) {
      vphase(t - 1, no);
      sync_odd();
      mphase(t, yes, yes);
      sync_even(t + 1);
    }
    vphase(nkb - 1, yes);
    sync_odd();
    mphase(nkb, no, yes);
  }
  __builtin_amdgcn_s_waitcnt(0);

  bf16* out = static_cast<bf16*>(a.out);
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float inv = 1.0f / l[qt][0];
    const int q = q0 + qt * 16 + lr;
    if (q >= a.T) continue;
    bf16* orow = out + ((size_t)b * a.T + q) * a.D + h * kDh;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      bf16x4 v;
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = static_cast<bf16>(o[d][qt][r] * inv);
      *reinterpret_cast<bf16x4*>(orow + d * 16 + g * 4) = v;
    }
  }
}

// ------------------------------------------------------------- fp32 attention
// One thread per query, online softmax over all keys (parity mode only).
template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  if (a.skip && *a.skip) return;
  const int bh = blockIdx.y;
  const int b = bh / a.H, h = bh % a.H;
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= a.T) return;
  const float* Q = static_cast<const float*>(a.q) + ((size_t)bh * a.Tpad + q) * DH;
  const float* Kg = static_cast<const float*>(a.k) + (size_t)bh * a.Tpad * DH;
  const float* Vt = static_cast<const float*>(a.vt) + (size_t)bh * DH * a.Tpad;
  float qv[DH], acc[DH];
  const float sc = rsqrtf((float)DH);
#pragma unroll
  for (int d = 0; d < DH; ++d) {
    qv[d] = Q[d] * sc;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j < a.T; ++j) {
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < DH; ++d) s += qv[d] * Kg[(size_t)j * DH + d];
    const float mn = fmaxf(m, s);
    const float corr = __expf(m - mn);
    const float p = __expf(s - mn);
    l = l * corr + p;
#pragma unroll
    for (int d = 0; d < DH; ++d) acc[d] = acc[d] * corr + p * Vt[(size_t)d * a.Tpad + j];
    m = mn;
  }
  float* orow = static_cast<float*>(a.out) + ((size_t)b * a.T + q) * a.D + h * DH;
  const float inv = 1.0f / l;
#pragma unroll
  for (int d = 0; d < DH; ++d) orow[d] = acc[d] * inv;
}

}  // namespace

hipError_t launch_qkv_relayout(const RelayoutArgs& a, bool bf16_mode, hipStream_t s) {
  dim3 grid((a.T + 63) / 64, a.H, a.B);
  if (a.dh == 64) {
    if (bf16_mode) launch_k(qkv_relayout_kernel<bf16, 64>, grid, 256, 0, s, a);
    else launch_k(qkv_relayout_kernel<float, 64>, grid, 256, 0, s, a);
  } else if (a.dh == 32) {
    if (bf16_mode) launch_k(qkv_relayout_kernel<bf16, 32>, grid, 256, 0, s, a);
    else launch_k(qkv_relayout_kernel<float, 32>, grid, 256, 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// grid for qt query tiles per wave and nw waves per block
// (qt, nw, st): query tiles of 16 per wave, waves per block, LDS stages of
// one 64-key K / V^T tile.  Only the instantiated combinations are accepted.
hipError_t launch_attention_cfg(const AttnArgs& a, int qt, int nw, int st, hipStream_t s, int form) {
  // every key tile but the last is fully inside [0, T), the last holds >= 1 key
  if (a.dh != kDh || a.T <= 0 || a.Tpad % kKB || a.T > a.Tpad || a.T <= a.Tpad - kKB) return hipErrorInvalidValue;
  if (form != ATTN_RUNNING && (!a.bounded || !(a.mref >= 0.f && a.mref <= kMaxBoundedRef))) return hipErrorInvalidValue;
  if (form == ATTN_PINGPONG) nw = 8;
  const int qb = qt * nw * 16;
  const dim3 grid((a.T + qb - 1) / qb, a.B * a.H);
  const int key = qt * 10000 + nw * 100 + st;
  switch (form) {
    case ATTN_PIPELINED:
      switch (key) {
        case 10404: launch_k(attn_bf16_bounded_kernel<1, 4, 4>, grid, 256, 0, s, a); break;
        case 20404: launch_k(attn_bf16_bounded_kernel<2, 4, 4>, grid, 256, 0, s, a); break;
        case 20403: launch_k(attn_bf16_bounded_kernel<2, 4, 3>, grid, 256, 0, s, a); break;
        default: return hipErrorInvalidValue;
      }
      break;
    case ATTN_PLAIN_KSPLIT:
      switch (key) {
        case 10402: launch_k(attn_bf16_kernel<1, 4, 2, true, 2>, grid, 512, 0, s, a); break;
        default: return hipErrorInvalidValue;
      }
      break;
    case ATTN_PLAIN:
      switch (key) {
        case 20402: launch_k(attn_bf16_kernel<2, 4, 2, true>, grid, 256, 0, s, a); break;
        case 20403: launch_k(attn_bf16_kernel<2, 4, 3, true>, grid, 256, 0, s, a); break;
        case 40802: launch_k(attn_bf16_kernel<4, 8, 2, true>, grid, 512, 0, s, a); break;
        default: return hipErrorInvalidValue;
      }
      break;
    case ATTN_PINGPONG:
      switch (key) {
        case 40804: launch_k(attn_bf16_pingpong_kernel<4, 4>, grid, 512, 0, s, a); break;
        case 20804: launch_k(attn_bf16_pingpong_kernel<2, 4>, grid, 512, 0, s, a); break;
        default: return hipErrorInvalidValue;
      }
      break;
    default:
      switch (key) {
        case 10404: launch_k(attn_bf16_kernel<1, 4, 4>, grid, 256, 0, s, a); break;
        case 20404: launch_k(attn_bf16_kernel<2, 4, 4>, grid, 256, 0, s, a); break;
        case 40403: launch_k(attn_bf16_kernel<4, 4, 3>, grid, 256, 0, s, a); break;
        case 10804: launch_k(attn_bf16_kernel<1, 8, 4>, grid, 512, 0, s, a); break;
        case 20804: launch_k(attn_bf16_kernel<2, 8, 4>, grid, 512, 0, s, a); break;
        case 20803: launch_k(attn_bf16_kernel<2, 8, 3>, grid, 512, 0, s, a); break;
        case 40402: launch_k(attn_bf16_kernel<4, 4, 2>, grid, 256, 0, s, a); break;
        case 20402: launch_k(attn_bf16_kernel<2, 4, 2>, grid, 256, 0, s, a); break;
        default: return hipErrorInvalidValue;
      }
  }
  return hipGetLastError();
}

float attention_score_bound(const float* q_g, const float* k_g) {
  // q = log2(e)/8 * g_q (.) qhat and k = g_k (.) khat with |qhat|, |khat| <= 8
  // (unit RMS over 64 dims), so |q.k| <= log2(e)/8 * 64 * max|g_q| * max|g_k|;
  // bf16 rounding of each element adds at most 2^-8 relative per operand
  float gq = 0.f, gk = 0.f;
  for (int i = 0; i < kDh; ++i) {
    gq = fmaxf(gq, fabsf(q_g[i]));
    gk = fmaxf(gk, fabsf(k_g[i]));
  }
  return kQLog2Scale * 64.0f * gq * gk * (1.0f + 1.0f / 128.0f) + 1e-3f;
}

hipError_t launch_attention(const AttnArgs& a, bool bf16_mode, hipStream_t s) {
  if (bf16_mode && a.bounded && a.variant != WAM_ATTN_RUNNING_MAX) {
    if (a.variant == WAM_ATTN_PINGPONG) return launch_attention_cfg(a, 4, 8, 4, s, ATTN_PINGPONG);
    // from a sweep at the workload shapes: long sequences with about two
    // blocks of 512 queries per CU take 8 waves of 64 queries; 4 waves of 32
    // queries when that fills the chip; short grids (T = 864, 12 heads: 168
    // blocks) two groups of 4 waves of 16 queries that split the keys (8.5
    // against 9.3 us), unless there are too few key tiles to split
    const bool big = a.T >= 4096 && (long)((a.T + 511) / 512) * a.B * a.H >= 384;
    const bool full = (long)((a.T + 127) / 128) * a.B * a.H >= 256;
    if (a.variant == WAM_ATTN_BOUNDED)
      return full ? launch_attention_cfg(a, 2, 4, 4, s, ATTN_PIPELINED) : launch_attention_cfg(a, 1, 4, 4, s, ATTN_PIPELINED);
    if (big) return launch_attention_cfg(a, 4, 8, 2, s, ATTN_PLAIN);
    if (full) return launch_attention_cfg(a, 2, 4, 2, s, ATTN_PLAIN);
    if (a.variant == WAM_ATTN_PLAIN || a.Tpad / kKB >= 4) return launch_attention_cfg(a, 1, 4, 2, s, ATTN_PLAIN_KSPLIT);
    return launch_attention_cfg(a, 1, 4, 4, s, ATTN_PIPELINED);
  }
  if (bf16_mode) {
    // 4 waves x 32 queries (two K/V stages) when that fills the chip, else
    // 4 waves x 16 queries
    const long blocks = (long)((a.T + 255) / 256) * a.B * a.H;
    if (blocks >= 256) return launch_attention_cfg(a, 2, 4, 2, s, ATTN_RUNNING);
    return launch_attention_cfg(a, 1, 4, 4, s, ATTN_RUNNING);
  }
  dim3 grid((a.T + 63) / 64, a.B * a.H);
  if (a.dh == 64) launch_k(attn_f32_kernel<64>, grid, 64, 0, s, a);
  else if (a.dh == 32) launch_k(attn_f32_kernel<32>, grid, 64, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace wam
