// Shared projections for small batches (decode: one token per request).
//
// With a few hundred rows every weight element is used by few rows, so the
// shared projections stream the weights from HBM, and the per-task LoRA work
// is a gather of each task's factors for the handful of rows it owns
// (Section 4.2 adapter handling, applied per task on the shared batch).
// Three kernels per projection group replace the large-tile GEMM:
//
//   gemm_skinny    Z[s, m, n] = sum over K range s of X[m, k] W[n, k]:
//                  256-row x BN-column tiles, two LDS stages fed by
//                  global_load_lds, K split so the grid covers the chip.
//                  Partials stay per split (fp32, no atomics), so results
//                  do not depend on scheduling.
//   shrink_split   P[c, m, slot + j] = sum over K chunk c of X[m, k] A_t[j, k]:
//                  one block per (task row tile, K chunk), so a task's A
//                  factors are read once, by many blocks at a time.
//   finalize       per row: U = bf16(s_t * sum_c P) rebuilt in LDS, then
//                  y = sum of the slices + U B_t^T + bias and the activation
//                  or residual epilogue, streamed one thread per 4 outputs
//                  (B_t rows read straight from the task's factor: the
//                  per-task adapter gather).
#include <algorithm>

#include "vfm_internal.h"

namespace {

typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// 128-byte LDS rows: logical 16-byte chunk kc of row r sits at chunk
// kc ^ ((r >> 1) & 7), which spreads the 16-row fragment reads over all banks.
__device__ __forceinline__ int swz(int row, int kc) { return kc ^ ((row >> 1) & 7); }

constexpr int SBM = 256, SBK = 64;

// ---------------------------------------------------------------------------
// Split-K GEMM, BN = 64 * NWN columns per block, 4 x NWN waves of 64 x 64.
//
// Every weight element is used by the few hundred rows of one tile only, so
// the weight stream comes from HBM at full latency while the activation
// columns are L2 hits.  Half of the waves load activation stages (one step
// ahead, two LDS stages), the other half weight stages (WST - 1 steps
// ahead, WST LDS stages): a wave's loads complete in issue order, so
// keeping the two streams in different waves lets the short-latency
// activation loads be waited on without waiting for the weight loads
// behind them.  All waves take part in the MFMA work.
// ---------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);   // vmcnt(N), lgkmcnt / expcnt not waited
}

template <int NWN, int WST>
__global__ __launch_bounds__(256 * NWN) void gemm_skinny_kernel(SkinnyArgs a) {
  // loader waves: half for each operand, except 192 columns (12 waves), whose
  // 256 activation rows need a power-of-two share (8 activation, 4 weight)
  constexpr int BN = 64 * NWN, NW = 4 * NWN, XW = NWN == 3 ? 8 : NW / 2, WW = NW - XW;
  constexpr int SA = SBM * SBK, SB = BN * SBK;
  constexpr int XR = SBM / (8 * XW), WR = BN / (8 * WW);    // 1 KB rounds per stage and loader wave
  static_assert(XR * 8 * XW == SBM && WR * 8 * WW == BN, "loader rounds");
  static_assert(WST == 3 || WST == 4, "weight stages");
  static_assert(WR * (WST - 2) < 16, "vmcnt range");
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * SA + WST * SB];
  // wave index in an SGPR, so the loader roles below are scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 3, wn = wave >> 2;
  const int ntn = (a.N + BN - 1) / BN;
  // consecutive blocks land on one XCD (the dispatcher deals block ids out
  // to the 8 XCDs in turn), so the blocks of one K split share that XCD's
  // L2 copy of the split's activation columns; the grid is padded to a
  // multiple of 8 and the padding blocks leave at once
  const int bx = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
  if (bx >= ntn * a.nsplit) return;
  const int tn = bx % ntn, split = bx / ntn;
  const int m0 = blockIdx.y * SBM, n0 = tn * BN;
  const int nkt = a.K / SBK;
  const int kt0 = (int)((int64_t)split * nkt / a.nsplit);
  const int kt1 = (int)((int64_t)(split + 1) * nkt / a.nsplit);
  const int nk = kt1 - kt0;

  // loader rows: wave lw of its operand fills rows lw * 8 + (lane >> 3) +
  // 8 * (loader waves) * i; the swizzle is applied on the global side, so
  // lane l writes chunk (l & 7) of its row (the chunk permutation is the
  // same for every round because 4 * loader waves is a multiple of 8)
  const bool xload = wave < XW;
  const int lw = xload ? wave : wave - XW;
  const int row0 = lw * 8 + (lane >> 3);
  const int kc0 = (lane & 7) ^ ((row0 >> 1) & 7);
  constexpr int MR = XR > WR ? XR : WR;
  const bf16* src[MR];
  if (xload) {
#pragma unroll
    for (int i = 0; i < XR; ++i)
      src[i] = (const bf16*)a.X + (int64_t)min(m0 + row0 + i * 8 * XW, a.M - 1) * a.ldx + kt0 * SBK + kc0 * 8;
  } else {
#pragma unroll
    for (int i = 0; i < WR; ++i) {
      const int n = min(n0 + row0 + i * 8 * WW, a.N - 1);
      const bool hi = a.W2 != nullptr && n >= a.n_half;
      src[i] = (const bf16*)(hi ? a.W2 : a.W) + (int64_t)(hi ? n - a.n_half : n) * a.K + kt0 * SBK + kc0 * 8;
    }
  }
  bf16* const Xs = smem;
  bf16* const Ws = smem + 2 * SA;
  auto issue_x = [&](int j) {   // step j of the block's K range into X stage j & 1
#pragma unroll
    for (int i = 0; i < XR; ++i)
      __builtin_amdgcn_global_load_lds((gptr_t)(src[i] + j * SBK),
                                       (lptr_t)(Xs + (j & 1) * SA + (i * XW + lw) * 512), 16, 0, 0);
  };
  // the weights are read once per forward: nontemporal (cache policy 2, nt)
  auto issue_w = [&](int j, int slot) {
#pragma unroll
    for (int i = 0; i < WR; ++i)
      __builtin_amdgcn_global_load_lds((gptr_t)(src[i] + j * SBK),
                                       (lptr_t)(Ws + slot * SB + (i * WW + lw) * 512), 16, 0, 2);
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (nk > 0) {
    if (xload) {
      issue_x(0);
    } else {
#pragma unroll
      for (int j = 0; j < WST - 1; ++j)
        if (j < nk) issue_w(j, j);
    }
    int ws = 0;                                   // W stage of step j
    for (int j = 0; j < nk; ++j) {
      // this wave's loads of step j have landed: the X loaders have nothing
      // newer in flight, the W loaders up to WST - 2 newer steps
      if (xload) {
        wait_vm<0>();
      } else {
        const int newer = min(nk - 1 - j, WST - 2);
        if constexpr (WST >= 4) {
          if (newer >= 2) wait_vm<2 * WR>();
          else if (newer == 1) wait_vm<WR>();
          else wait_vm<0>();
        } else {
          if (newer >= 1) wait_vm<WR>();
          else wait_vm<0>();
        }
      }
      __builtin_amdgcn_s_barrier();
      // every wave is past step j - 1, whose X stage and W stage are free
      if (xload) {
        if (j + 1 < nk) issue_x(j + 1);
      } else {
        if (j + WST - 1 < nk) issue_w(j + WST - 1, ws == 0 ? WST - 1 : ws - 1);
      }
      const bf16* As = Xs + (j & 1) * SA;
      const bf16* Bs = Ws + ws * SB;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int kc = kk * 4 + (lane >> 4);
        bf16x8 wf[4], xf[4];
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
          const int r = wn * 64 + ni * 16 + (lane & 15);
          wf[ni] = *reinterpret_cast<const bf16x8*>(Bs + r * SBK + swz(r, kc) * 8);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
          const int r = wm * 64 + mi * 16 + (lane & 15);
          xf[mi] = *reinterpret_cast<const bf16x8*>(As + r * SBK + swz(r, kc) * 8);
        }
#pragma unroll
        for (int mi = 0; mi < 4; ++mi)
#pragma unroll
          for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = mfma16(wf[ni], xf[mi], acc[mi][ni]);
      }
      ws = ws == WST - 1 ? 0 : ws + 1;
    }
  }
  // lane holds D[n = 4 * (lane >> 4) + i][m = lane & 15] of each 16 x 16 block
  float* Zs = a.Z + (int64_t)split * a.M * a.N;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi) {
    const int m = m0 + wm * 64 + mi * 16 + (lane & 15);
    if (m >= a.M) continue;
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
      const int n = n0 + wn * 64 + ni * 16 + 4 * (lane >> 4);
      if (n >= a.N) continue;
      *reinterpret_cast<float4*>(Zs + (int64_t)m * a.N + n) =
          make_float4(acc[mi][ni][0], acc[mi][ni][1], acc[mi][ni][2], acc[mi][ni][3]);
    }
  }
}

// ---------------------------------------------------------------------------
// Split-K segmented shrink.  Each wave owns 16 rows of the tile and every
// projection of the group; A rows feed the MFMA A slot, X rows the B slot.
// ---------------------------------------------------------------------------
template <int NP, int NSUB>
__global__ __launch_bounds__(256) void shrink_split_kernel(Plan pl, ShrinkSplitArgs a) {
  __shared__ int s_task;
  const int tile = blockIdx.x, c = blockIdx.y;
  const int t = block_tile_task(pl, tile, &s_task);
  const int r0 = pl.seg_row[t] + (tile - pl.rtile_off[t]) * VFM_ROW_TILE;
  const int r1 = min(r0 + VFM_ROW_TILE, pl.seg_row[t + 1]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rank = min(a.rank[t], NSUB * 16);
  const int m = r0 + wave * 16 + (lane & 15);
  const int k0 = c * a.kchunk, k1 = min(k0 + a.kchunk, a.K);
  const bf16* X = (const bf16*)a.X;
  f32x4 acc[NP][NSUB];
#pragma unroll
  for (int pp = 0; pp < NP; ++pp)
#pragma unroll
    for (int s = 0; s < NSUB; ++s) acc[pp][s] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (rank > 0 && r0 + wave * 16 < r1) {
    const bf16* xrow = X + (int64_t)min(m, r1 - 1) * a.ldx + 8 * (lane >> 4);
    const bf16* arow[NP][NSUB];
    bool on[NSUB];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) on[s] = s * 16 + (lane & 15) < rank;
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
      const bf16* At = (const bf16*)a.A[pp][t];
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
        arow[pp][s] = At + (int64_t)min(s * 16 + (lane & 15), rank - 1) * a.K + 8 * (lane >> 4);
    }
#pragma unroll 4
    for (int k = k0; k < k1; k += 32) {
      const bf16x8 xf = *reinterpret_cast<const bf16x8*>(xrow + k);
#pragma unroll
      for (int pp = 0; pp < NP; ++pp)
#pragma unroll
        for (int s = 0; s < NSUB; ++s) {
          bf16x8 af = *reinterpret_cast<const bf16x8*>(arow[pp][s] + k);
          if (!on[s]) af = bf16x8{};
          acc[pp][s] = mfma16(af, xf, acc[pp][s]);
        }
    }
  }
  if (m < r1) {
    float* P = a.P + ((int64_t)c * pl.T + m) * a.ldp;
#pragma unroll
    for (int pp = 0; pp < NP; ++pp)
#pragma unroll
      for (int s = 0; s < NSUB; ++s)
        *reinterpret_cast<float4*>(P + a.ucol[pp] + s * 16 + 4 * (lane >> 4)) =
            make_float4(acc[pp][s][0], acc[pp][s][1], acc[pp][s][2], acc[pp][s][3]);
  }
}

// ---------------------------------------------------------------------------
// Finalize: sum of the partial slices (fixed order) + the row's LoRA
// difference (fin_lora_delta, from the split shrink's partials) + bias +
// epilogue.  Block (column range, row): the row's U is rebuilt once in LDS,
// then each thread takes 4 output columns; every load is independent of the
// others, so the kernel streams the partials.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void finalize_kernel(FinalizeArgs a) {
  __shared__ float Us[3 * VFM_MAX_RANK], red[256];
  __shared__ float rcs[64], rsn[64];          // the row's rotary angles (head_dim / 2 <= 64)
  // Block b takes (column block, row) number (b % 8) * per + b / 8, rows
  // fastest: consecutive blocks of one XCD (one L2) take consecutive rows of
  // one column block, so a task's B rows, read again for its next rows, come
  // from that XCD's L2 instead of beyond it.
  const int ncb = (a.N / 4 + 255) / 256;
  const int per = gridDim.x / 8;
  const int lid = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (lid >= ncb * a.M) return;               // block-uniform
  const int m = lid % a.M, cb = lid / a.M;
  int t = 0, r = 0;
  FinB bp = {};
  if (a.lora.enabled) {                       // block-uniform
    t = a.lora.row_task[m];
    bp = fin_lora_bptrs(a.lora, t);
    r = fin_lora_u(a.lora, m, Us, red);
  }
  if (a.rope.on) {                            // block-uniform: the row's angles, as launch_rope
    const int half = a.rope.head_dim >> 1;
    if (threadIdx.x < half) {
      const float inv = exp2f(-(2.0f * (float)threadIdx.x / (float)a.rope.head_dim) * a.rope.log2_theta);
      float sn, cs;
      sincosf((float)a.rope.pl.pos[m] * inv, &sn, &cs);
      rcs[threadIdx.x] = cs;
      rsn[threadIdx.x] = sn;
    }
    __syncthreads();
  }
  const int n = (cb * 256 + threadIdx.x) * 4;
  if (n >= a.N) return;
  const bool swiglu = a.epi == EPI_SWIGLU;
  const int nz = swiglu ? 2 * a.N : a.N;   // columns of Z
  const int64_t zs = (int64_t)a.M * nz;
  const float* z = a.Z + (int64_t)m * nz + n;
  float4 v = sum_slices(z, zs, a.nslices);
  if (a.lora.enabled) {
    if (swiglu) {
      add4(v, fin_lora_delta(a.lora, bp, r, 0, n, Us));
    } else {
      const int slot = min(n / a.lora.slot_width, 2);
      add4(v, fin_lora_delta(a.lora, bp, r, slot, n - slot * a.lora.slot_width, Us));
    }
  }
  if (a.bias && !swiglu) {
    const bf16x4 bv = *reinterpret_cast<const bf16x4*>((const bf16*)a.bias + n);
    v.x += (float)bv[0]; v.y += (float)bv[1]; v.z += (float)bv[2]; v.w += (float)bv[3];
  }
  if (a.epi == EPI_RESID) {
    float4* xo = reinterpret_cast<float4*>((float*)a.out + (int64_t)m * a.ldo + n);
    float4 xv = *xo;
    add4(xv, v);
    *xo = xv;
    return;
  }
  if (a.rope.on && n < 2 * a.rope.d) {        // q and k columns (whole waves: d % 256 == 0)
    // rotate-half: column i of a head pairs with column i + head_dim / 2,
    // held head_dim / 8 lanes away (4 columns per lane)
    const int dh = a.rope.head_dim, half = dh >> 1;
    const int cin = n % dh;
    float4 pv;
    pv.x = __shfl_xor(v.x, dh / 8, 64);
    pv.y = __shfl_xor(v.y, dh / 8, 64);
    pv.z = __shfl_xor(v.z, dh / 8, 64);
    pv.w = __shfl_xor(v.w, dh / 8, 64);
    const bool second = cin >= half;
    const int i0 = second ? cin - half : cin;
    float x4[4] = {v.x, v.y, v.z, v.w};
    const float p4[4] = {pv.x, pv.y, pv.z, pv.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float cs = rcs[i0 + c], sn = rsn[i0 + c];
      x4[c] = second ? p4[c] * sn + x4[c] * cs : x4[c] * cs - p4[c] * sn;
    }
    v = make_float4(x4[0], x4[1], x4[2], x4[3]);
  }
  const float g4[4] = {v.x, v.y, v.z, v.w};
  float u4[4] = {0.f, 0.f, 0.f, 0.f};
  if (swiglu) {
    float4 u = sum_slices(z + a.N, zs, a.nslices);
    if (a.lora.enabled) add4(u, fin_lora_delta(a.lora, bp, r, 1, n, Us));
    u4[0] = u.x; u4[1] = u.y; u4[2] = u.z; u4[3] = u.w;
  }
  bf16x4 o;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float y = g4[c];
    if (swiglu) y = silu_fast(y) * u4[c];
    else if (a.epi == EPI_GELU) y = gelu_fast(y);
    o[c] = (bf16)y;
  }
  *reinterpret_cast<bf16x4*>((bf16*)a.out + (int64_t)m * a.ldo + n) = o;
  if (a.rope.on && a.rope.kc != nullptr && n >= a.rope.d) {   // the row's k (rotated) and v to its slot
    const int dd = a.rope.d, dh = a.rope.head_dim;
    const bool isv = n >= 2 * dd;
    const int cc = isv ? n - 2 * dd : n - dd;
    const int hh = cc / dh;
    const int64_t slot = kv_slot(a.rope.pl, a.rope.kp, a.rope.pl.row_req[m], a.rope.pl.pos[m]);
    bf16* dst = (isv ? a.rope.vc : a.rope.kc) + ((int64_t)hh * a.rope.kv_slots + slot) * dh + (cc - hh * dh);
    *reinterpret_cast<bf16x4*>(dst) = o;
  }
}

// Column-tile width and K split of the small-batch GEMM for an N x K
// weight: for each tile width (128, 192, 256 columns) K is split until one
// row tile fills the chip once (one block per CU), at most 6 ways for wide
// weights (N >= 8192) so the fp32 partials stay below the weight bytes; the
// width whose blocks each stream the fewest weight bytes wins (the 7B
// gate/up weight: 230 blocks of 192 columns instead of 172 of 256).  The
// split depends on the weight shape only, never on the batch, so a row's
// result does not depend on the other rows.
void skinny_shape(int N, int K, int* bn, int* nsplit) {
  const int nkt = K / SBK;
  const bool wide = N >= 8192;
  const int cap = wide ? 6 : 16;
  // the tile width whose one round of blocks streams the fewest weight
  // steps per block (rounds x width x K steps of a split); ties go to fewer
  // splits (fewer partial bytes)
  long best = -1;
  for (const int b : {128, 192, 256}) {
    const int tiles = (N + b - 1) / b;
    const int ns = std::max(1, std::min(std::min(256 / tiles, cap), nkt));
    const long rounds = ((long)tiles * ns + 255) / 256;
    const long cost = rounds * b * ((nkt + ns - 1) / ns);
    if (best < 0 || cost < best || (cost == best && ns < *nsplit)) {
      best = cost;
      *bn = b;
      *nsplit = ns;
    }
  }
}

}  // namespace

int skinny_splits(int N, int K) {
  int bn, ns;
  skinny_shape(N, K, &bn, &ns);
  return ns;
}

hipError_t launch_gemm_skinny(const SkinnyArgs& a0, hipStream_t s) {
  if (a0.M == 0) return hipSuccess;
  SkinnyArgs a = a0;
  int bn;
  skinny_shape(a.N, a.K, &bn, &a.nsplit);
  const int ntn = (a.N + bn - 1) / bn;
  dim3 grid((ntn * a.nsplit + 7) & ~7, (a.M + SBM - 1) / SBM);
  if (bn == 128)
    hipLaunchKernelGGL((gemm_skinny_kernel<2, 4>), grid, dim3(512), 0, s, a);
  else if (bn == 192)
    hipLaunchKernelGGL((gemm_skinny_kernel<3, 4>), grid, dim3(768), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_skinny_kernel<4, 3>), grid, dim3(1024), 0, s, a);
  return hipGetLastError();
}

// K chunks of the split shrink: fixed 256-column chunks (the last one
// ragged), independent of the batch for the same reason as the GEMM split.
int shrink_chunks(int K) { return (K + 255) / 256; }

hipError_t launch_shrink_split(const Plan& pl, const ShrinkSplitArgs& a0, hipStream_t s) {
  if (pl.n_rtiles == 0 || a0.n_proj == 0) return hipSuccess;
  ShrinkSplitArgs a = a0;
  a.kchunk = 256;
  dim3 grid(pl.n_rtiles, a.kchunks);
#define VFM_SS(NP_, NS_) hipLaunchKernelGGL((shrink_split_kernel<NP_, NS_>), grid, dim3(256), 0, s, pl, a)
  // only the sub-tiles the table's largest rank reaches: 1 (rank <= 16), 2 (<= 32) or 4
#define VFM_SS_NP(NS_) do { if (a.n_proj == 1) VFM_SS(1, NS_); else if (a.n_proj == 2) VFM_SS(2, NS_); else VFM_SS(3, NS_); } while (0)
  if (a.nsub <= 1) VFM_SS_NP(1);
  else if (a.nsub == 2) VFM_SS_NP(2);
  else VFM_SS_NP(4);
#undef VFM_SS_NP
#undef VFM_SS
  return hipGetLastError();
}

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  const int ncb = (a.N / 4 + 255) / 256;
  hipLaunchKernelGGL(finalize_kernel, dim3(((int64_t)ncb * a.M + 7) / 8 * 8), dim3(256), 0, s, a);
  return hipGetLastError();
}
