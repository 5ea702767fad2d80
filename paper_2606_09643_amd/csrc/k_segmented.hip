// Per-task segmented kernels: LoRA shrink (a4), LoRA expand (the standalone
// vfm_lora_apply), and the per-task linear heads (a12).
//
// Rows are in plan order, so every task owns one contiguous segment of rows
// (and of requests).  Work is split into VFM_ROW_TILE-row tiles that never
// cross a task boundary (the plan's rtile_off), so a skewed task mix (a Zipf
// head task holding a third of the rows) still spreads over many blocks, and
// each block reads exactly one task's factors.  The task's A / B / head
// weights are gathered through the per-task pointer tables, so attaching or
// removing a task is a pointer update (paper Section 4.1 task extensions;
// Table 1 attach_adapter / remove_adapter).
//
// bf16: v_mfma_f32_16x16x32_bf16 with operands read straight from global
// memory (16-byte per-lane loads); the adapter factor feeds the MFMA A slot,
// the activation rows the B slot, so each lane ends with 4 consecutive
// output columns of one row.  fp32: plain per-thread dot products.
#include "vfm_internal.h"

namespace {

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Locate the task and row range of segmented tile `bid`.
__device__ inline void tile_rows(const Plan& pl, int bid, int& t, int& r0, int& r1) {
  t = upper_index(pl.rtile_off, pl.n_tasks + 1, bid);
  r0 = pl.seg_row[t] + (bid - pl.rtile_off[t]) * VFM_ROW_TILE;
  r1 = min(r0 + VFM_ROW_TILE, pl.seg_row[t + 1]);
}

// ---------------------------------------------------------------------------
// shrink: U[m, ucol + j] = s_t * X[m, :] . A_t[j, :]   (j < rpad, zero past r_t)
// ---------------------------------------------------------------------------
typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;
__device__ __attribute__((aligned(16))) bf16 g_seg_zero[8];  // zero-initialised at load

// The task owning tile `tile` of the tiling that cuts each task's rows into
// ceil(rows_t / ROWS) tiles, in task order, and the tile's first row; one
// wave counts the tiles (each lane a contiguous run of tasks, then a prefix
// over the lanes) and the lane holding the tile finds it.  Returns false
// (block-uniform) past the last tile.  sl: 2 ints of LDS.
template <int ROWS>
__device__ inline bool rows_tile_task(const Plan& pl, int tile, int* sl, int* t_out, int* r0_out) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x, n = pl.n_tasks;
    if (lane == 0) sl[0] = -1;
    const int per = (n + 63) / 64;
    const int t0 = min(lane * per, n), t1 = min(t0 + per, n);
    int cnt = 0;
    for (int t = t0; t < t1; ++t) cnt += (pl.seg_row[t + 1] - pl.seg_row[t] + ROWS - 1) / ROWS;
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
    int off = incl - cnt;
    if (tile >= off && tile < incl) {
      for (int t = t0; t < t1; ++t) {
        const int nt = (pl.seg_row[t + 1] - pl.seg_row[t] + ROWS - 1) / ROWS;
        if (tile < off + nt) {
          sl[0] = t;
          sl[1] = pl.seg_row[t] + (tile - off) * ROWS;
          break;
        }
        off += nt;
      }
    }
  }
  __syncthreads();
  *t_out = sl[0];
  *r0_out = sl[1];
  return *t_out >= 0;
}

template <int NP, int NSUB, int NWV>
__global__ __launch_bounds__(64 * NWV) void shrink_bf16_kernel(Plan pl, ShrinkArgs a) {
  // One block per tile of 16 * NWV rows of one task (the plan's 64-row tiles
  // with 4 waves; 96-row tiles with 6 when the batch has more 64-row tiles
  // than CUs, so one round of blocks covers it); wave w owns 16 rows and
  // every projection of the group, so each row is read once for all of
  // them.  Each 64-column chunk of the task's A rows (shared by the waves)
  // and of the tile's activation rows goes through an LDS ring of NST stages
  // fed by global_load_lds: every wave-wide load moves 8 whole 128-byte rows,
  // and NST - 1 chunks are in flight while one is consumed.  A rows past the
  // rank come from a zero page; only the NSUB 16-row sub-tiles that the
  // largest rank reaches are computed.  LDS rows are 128 B with chunk
  // swizzle kc ^ ((row >> 1) & 7); a stage holds AR A rows, then the tile's
  // rows, then padding to whole block passes.  A row's sums are the same
  // MFMAs in the same order for either tile size.
  static_assert(NWV == 4 || NWV == 6, "the swizzle repeats every block pass for an even wave count");
  constexpr int ROWS = 16 * NWV;                // activation rows per block
  constexpr int AR = NP * NSUB * 16;            // A rows the MFMAs read per chunk
  constexpr int PR = 8 * NWV;                   // LDS rows one block pass of 16-byte loads fills
  constexpr int SR = (AR + ROWS + PR - 1) / PR * PR;   // LDS rows per stage
  constexpr int NST = 4;
  constexpr int ND = SR / PR;                   // 16-byte pieces per thread and chunk
  static_assert(NWV != 4 || ROWS == VFM_ROW_TILE, "the plan's row tiles");
  // one LDS object (the task slot sits past the ring): with a second one the
  // compiler would wait for the ring's DMA before every fragment read
  __shared__ __attribute__((aligned(16))) bf16 As[NST][SR * 64 + 8];
  int* const sl = reinterpret_cast<int*>(&As[NST - 1][SR * 64]);
  const int tile = blockIdx.x;
  int t, r0;
  if (NWV == 4) {
    t = block_tile_task(pl, tile, sl);
    r0 = pl.seg_row[t] + (tile - pl.rtile_off[t]) * VFM_ROW_TILE;
  } else if (!rows_tile_task<ROWS>(pl, tile, sl, &t, &r0)) {
    return;                                     // block-uniform: past the last tile
  }
  const int r1 = min(r0 + ROWS, pl.seg_row[t + 1]);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rank = min(a.rank[t], NSUB * 16) & ~7;
  const float sc = a.scale[t];
  const bf16* X = (const bf16*)a.X;
  bf16* U = (bf16*)a.U;
  const int m = r0 + wave * 16 + (lane & 15);
  f32x4 acc[NP][NSUB];
#pragma unroll
  for (int pp = 0; pp < NP; ++pp)
#pragma unroll
    for (int s2 = 0; s2 < NSUB; ++s2) acc[pp][s2] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (rank > 0) {   // block-uniform
    const bf16* src0[ND];
    const int prow0 = wave * 8 + (lane >> 3);
    const int kcl = (lane & 7) ^ ((prow0 >> 1) & 7);   // same for prow0 + PR i
#pragma unroll
    for (int i = 0; i < ND; ++i) {
      const int row = prow0 + i * PR;
      if (row < AR) {                                   // row = (pp*NSUB + s2)*16 + j
        const int pp = row / (NSUB * 16), j = row % (NSUB * 16);
        src0[i] = j < rank ? (const bf16*)a.A[pp][t] + (int64_t)j * a.K + kcl * 8 : nullptr;
      } else if (row < AR + ROWS) {                     // rows past the tile's end re-read its last row
        src0[i] = X + (int64_t)min(r0 + row - AR, r1 - 1) * a.ldx + kcl * 8;
      } else {
        src0[i] = nullptr;                              // padding rows (never read)
      }
    }
    const int nc = a.K / 64;
    // every chunk index past the end re-reads the last chunk, so each step
    // issues the same ND loads and one wait count holds throughout
    auto issue = [&](int c, int st) {
      const int cc = min(c, nc - 1);
#pragma unroll
      for (int i = 0; i < ND; ++i) {
        const bf16* src = src0[i] ? src0[i] + cc * 64 : g_seg_zero;
        __builtin_amdgcn_global_load_lds((gptr_t)src, (lptr_t)(&As[st][(i * NWV + wave) * 512]), 16, 0, 0);
      }
    };
#pragma unroll
    for (int i = 0; i < NST - 1; ++i) issue(i, i);
    for (int c0 = 0; c0 < nc; c0 += NST) {
#pragma unroll
      for (int j = 0; j < NST; ++j) {
        const int c = c0 + j;
        if (c >= nc) break;
        // chunk c landed once at most (NST - 2) later groups are outstanding
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((NST - 2) * ND) : "memory");
        __builtin_amdgcn_s_barrier();     // every wave's part is in LDS; stage (c-1) is free
        issue(c + NST - 1, (j + NST - 1) % NST);
        const bf16* Ab = As[j];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const int kc = kk * 4 + (lane >> 4);
          const int xr = AR + wave * 16 + (lane & 15);
          const bf16x8 xf = *reinterpret_cast<const bf16x8*>(Ab + xr * 64 + ((kc ^ ((xr >> 1) & 7)) * 8));
#pragma unroll
          for (int pp = 0; pp < NP; ++pp)
#pragma unroll
            for (int s2 = 0; s2 < NSUB; ++s2) {
              const int r = (pp * NSUB + s2) * 16 + (lane & 15);
              const bf16x8 af = *reinterpret_cast<const bf16x8*>(Ab + r * 64 + ((kc ^ ((r >> 1) & 7)) * 8));
              acc[pp][s2] = mfma16(af, xf, acc[pp][s2]);
            }
        }
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // nothing lands after the block ends
  }
  if (m < r1) {
#pragma unroll
    for (int pp = 0; pp < NP; ++pp)
#pragma unroll
      for (int s2 = 0; s2 < NSUB; ++s2) {
        bf16x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (bf16)(acc[pp][s2][i] * sc);
        *reinterpret_cast<bf16x4*>(U + (int64_t)m * a.ldu + a.ucol[pp] + s2 * 16 + 4 * (lane >> 4)) = o;
      }
    // the slot's columns past the computed sub-tiles (past every task's rank)
    for (int pp = 0; pp < NP; ++pp)
      for (int s2 = NSUB; s2 < a.rpad / 16; ++s2)
        *reinterpret_cast<bf16x4*>(U + (int64_t)m * a.ldu + a.ucol[pp] + s2 * 16 + 4 * (lane >> 4)) = bf16x4{};
  }
}

// fp32 shrink: one block per (16-row group of a segmented tile, projection);
// thread (row r, column jj) accumulates U[r, jj + 16 q] for q < rpad / 16
// over the whole of K with 16-byte loads (the row's loads are shared by its
// 16 threads through L1).  No LDS, no barrier.
__global__ __launch_bounds__(256) void shrink_f32_stream_kernel(Plan pl, ShrinkArgs a) {
  __shared__ int tslot;
  const int tile = blockIdx.x >> 2, grp = blockIdx.x & 3, p = blockIdx.y;
  const int t = block_tile_task(pl, tile, &tslot);
  const int r0 = pl.seg_row[t] + (tile - pl.rtile_off[t]) * VFM_ROW_TILE + grp * 16;
  const int r1 = min(pl.seg_row[t] + (tile - pl.rtile_off[t] + 1) * VFM_ROW_TILE, pl.seg_row[t + 1]);
  if (r0 >= r1) return;
  const int r = threadIdx.x >> 4, jj = threadIdx.x & 15;
  const int m = r0 + r;
  const int rank = min(a.rank[t], a.rpad) & ~7;
  const int nq = a.rpad / 16;                         // outputs per thread (2 or 4)
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  if (rank > 0 && m < r1) {
    const float* xr = (const float*)a.X + (int64_t)m * a.ldx;
    const float* At = (const float*)a.A[p][t];
    for (int k = 0; k < a.K; k += 4) {
      const float4 xv = *reinterpret_cast<const float4*>(xr + k);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = jj + 16 * q;
        if (q < nq && j < rank) {
          const float4 av = *reinterpret_cast<const float4*>(At + (int64_t)j * a.K + k);
          acc[q] = fmaf(xv.x, av.x, acc[q]);
          acc[q] = fmaf(xv.y, av.y, acc[q]);
          acc[q] = fmaf(xv.z, av.z, acc[q]);
          acc[q] = fmaf(xv.w, av.w, acc[q]);
        }
      }
    }
  }
  if (m >= r1) return;
  const float sc = a.scale[t];
  float* U = (float*)a.U;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (q < nq) U[(int64_t)m * a.ldu + a.ucol[p] + jj + 16 * q] = acc[q] * sc;
}

__global__ __launch_bounds__(256) void shrink_f32_kernel(Plan pl, ShrinkArgs a) {
  // One block per (row tile, projection).  K is walked in 32-column chunks
  // staged in LDS (the tile's rows and the task's A rows); thread (row i,
  // group g) accumulates rpad/4 outputs of row i from LDS.
  constexpr int KC = 32;
  __shared__ float xs[VFM_ROW_TILE][KC + 1];
  __shared__ float as[VFM_MAX_RANK][KC + 1];
  int t, r0, r1;
  tile_rows(pl, blockIdx.x, t, r0, r1);
  const int p = blockIdx.y;
  const int rank = min(a.rank[t], a.rpad) & ~7;
  const float sc = a.scale[t];
  const float* X = (const float*)a.X;
  const float* At = rank > 0 ? (const float*)a.A[p][t] : nullptr;
  float* U = (float*)a.U;
  const int rows = r1 - r0;
  const int i = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int jn = a.rpad / 4;                  // outputs per thread (8 or 16)
  float acc[VFM_MAX_RANK / 4];
#pragma unroll
  for (int q = 0; q < VFM_MAX_RANK / 4; ++q) acc[q] = 0.f;
  if (rank > 0) {
    for (int k0 = 0; k0 < a.K; k0 += KC) {
      for (int e = threadIdx.x; e < VFM_ROW_TILE * KC; e += 256) {
        const int r = e / KC, k = e % KC;
        xs[r][k] = r < rows ? X[(int64_t)(r0 + r) * a.ldx + k0 + k] : 0.f;
      }
      for (int e = threadIdx.x; e < a.rpad * KC; e += 256) {
        const int j = e / KC, k = e % KC;
        as[j][k] = j < rank ? At[(int64_t)j * a.K + k0 + k] : 0.f;
      }
      __syncthreads();
#pragma unroll 4
      for (int k = 0; k < KC; ++k) {
        const float xv = xs[i][k];
#pragma unroll
        for (int q = 0; q < VFM_MAX_RANK / 4; ++q)
          if (q < jn) acc[q] = fmaf(xv, as[g * jn + q][k], acc[q]);
      }
      __syncthreads();
    }
  }
  if (i < rows) {
#pragma unroll
    for (int q = 0; q < VFM_MAX_RANK / 4; ++q)
      if (q < jn) U[(int64_t)(r0 + i) * a.ldu + a.ucol[p] + g * jn + q] = acc[q] * sc;
  }
}

// ---------------------------------------------------------------------------
// expand: Y[m, n] += U[m, ucol + :r] . B_t[n, :r]     (fp32 Y)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void expand_bf16_kernel(Plan pl, ExpandArgs a) {
  int t, r0, r1;
  tile_rows(pl, blockIdx.x, t, r0, r1);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rank = min(a.rank[t], a.max_rank) & ~7;
  const int wr0 = r0 + wave * 16;
  if (rank <= 0 || wr0 >= r1) return;
  const int n0 = blockIdx.y * 64;
  const bf16* U = (const bf16*)a.U;
  const bf16* Bt = (const bf16*)a.B[t];
  f32x4 acc[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) acc[s] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int m = wr0 + (lane & 15);
  for (int kk = 0; kk < rank; kk += 32) {
    const int kof = kk + 8 * (lane >> 4);
    bf16x8 xf = {};
    if (m < r1 && kof < rank) xf = *reinterpret_cast<const bf16x8*>(U + (int64_t)m * a.ldu + a.ucol + kof);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int n = n0 + s * 16 + (lane & 15);
      bf16x8 wf = {};
      if (n < a.N && kof < rank) wf = *reinterpret_cast<const bf16x8*>(Bt + (int64_t)n * rank + kof);
      acc[s] = mfma16(wf, xf, acc[s]);
    }
  }
  if (m >= r1) return;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int n = n0 + s * 16 + 4 * (lane >> 4);
    if (n >= a.N) continue;
    float4* dst = reinterpret_cast<float4*>(a.Y + (int64_t)m * a.ldy + n);
    float4 o = *dst;
    o.x += acc[s][0]; o.y += acc[s][1]; o.z += acc[s][2]; o.w += acc[s][3];
    *dst = o;
  }
}

__global__ __launch_bounds__(256) void expand_f32_kernel(Plan pl, ExpandArgs a) {
  int t, r0, r1;
  tile_rows(pl, blockIdx.x, t, r0, r1);
  const int rank = min(a.rank[t], a.max_rank) & ~7;
  if (rank <= 0) return;
  const int n0 = blockIdx.y * 64;
  const float* U = (const float*)a.U;
  const float* Bt = (const float*)a.B[t];
  for (int e = threadIdx.x; e < (r1 - r0) * 64; e += 256) {
    const int m = r0 + e / 64, n = n0 + e % 64;
    if (n >= a.N) continue;
    float s = 0.f;
    for (int j = 0; j < rank; ++j) s += U[(int64_t)m * a.ldu + a.ucol + j] * Bt[(int64_t)n * rank + j];
    a.Y[(int64_t)m * a.ldy + n] += s;
  }
}

// ---------------------------------------------------------------------------
// heads: out[out_off[order[p]] + n] = pooled[p] . W_t[n] + b_t[n]
// One block per (task, 64-column chunk); the block walks the task's
// requests 16 at a time; each wave owns 16 of the 64 columns.
// ---------------------------------------------------------------------------
// Head GEMMs of one task's requests.  HID: the MLP heads' first layer,
// hid[p, n] = act(pooled[p] . W1_t[n] + b1_t[n]) for tasks with an MLP head;
// otherwise the output layer, out = in[p] . W_t[n] + b_t[n] with `in` the
// pooled row (linear head) or the hidden row (MLP head).
template <bool HID>
__global__ __launch_bounds__(256) void heads_bf16_kernel(Plan pl, const bf16* __restrict__ pooled,
                                                         int d, vfm_head_table h, bf16* __restrict__ hid,
                                                         float* __restrict__ out) {
  __shared__ f32x4 red[4][64];
  const int t = blockIdx.x;
  const bool mlp = h.W1 != nullptr && h.W1[t] != nullptr;
  if (HID && !mlp) return;                            // block-uniform
  const int n_out = HID ? h.hidden : h.n_out[t];
  const int n0 = blockIdx.y * 64;
  const int p0 = pl.seg_req[t], p1 = pl.seg_req[t + 1];
  if (p0 == p1 || n0 >= n_out) return;                // block-uniform
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bf16* Wt = (const bf16*)(HID ? h.W1[t] : h.W[t]);
  const bf16* bt = HID ? (h.b1 ? (const bf16*)h.b1[t] : nullptr) : (h.b ? (const bf16*)h.b[t] : nullptr);
  const bool from_hid = !HID && mlp;
  const int K = from_hid ? h.hidden : d;
  const bf16* in = from_hid ? hid : pooled;
  // at most 16 outputs left in this block: the 4 waves split K over the same
  // 16 rows and add their sums in wave order; otherwise each wave owns 16 rows
  const bool ksplit = n_out - n0 <= 16 && K % 128 == 0;
  const int rb = ksplit ? n0 : n0 + wave * 16;        // the wave's first output row
  const int kq = ksplit ? K / 4 : K;                  // K per wave
  const int kb = ksplit ? wave * kq : 0;
  const int nrow = rb + (lane & 15);
  const bf16* wrow = Wt + (int64_t)min(nrow, n_out - 1) * K + kb + 8 * (lane >> 4);
  for (int pb = p0; pb < p1; pb += 16) {
    const int p = pb + (lane & 15);
    const bf16* xrow = in + (int64_t)min(p, p1 - 1) * K + kb + 8 * (lane >> 4);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int k = 0; k < kq; k += 32) {
      const bf16x8 wf = *reinterpret_cast<const bf16x8*>(wrow + k);
      const bf16x8 xf = *reinterpret_cast<const bf16x8*>(xrow + k);
      acc = mfma16(wf, xf, acc);
    }
    if (ksplit) {
      red[wave][lane] = acc;
      __syncthreads();
      if (wave == 0) {
#pragma unroll
        for (int w = 1; w < 4; ++w) {
          const f32x4 u = red[w][lane];
          acc[0] += u[0]; acc[1] += u[1]; acc[2] += u[2]; acc[3] += u[3];
        }
      }
      __syncthreads();                                // red is reused by the next group
    }
    if (p < p1 && (!ksplit || wave == 0)) {
      if (HID) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int n = rb + 4 * (lane >> 4) + i;
          const float v = acc[i] + (bt ? (float)bt[n] : 0.f);
          hid[(int64_t)p * h.hidden + n] = (bf16)(h.act == VFM_ACT_RELU ? fmaxf(v, 0.f) : gelu_fast(v));
        }
      } else {
        const int req = pl.order[p];
        const int lim = min(n_out, pl.out_off[req + 1] - pl.out_off[req]);
        float* o = out + pl.out_off[req];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int n = rb + 4 * (lane >> 4) + i;
          if (n < lim) o[n] = acc[i] + (bt ? (float)bt[n] : 0.f);
        }
      }
    }
  }
}

template <bool HID>
__global__ __launch_bounds__(256) void heads_f32_kernel(Plan pl, const float* __restrict__ pooled,
                                                        int d, vfm_head_table h, float* __restrict__ hid,
                                                        float* __restrict__ out) {
  const int t = blockIdx.x;
  const bool mlp = h.W1 != nullptr && h.W1[t] != nullptr;
  if (HID && !mlp) return;
  const int n_out = HID ? h.hidden : h.n_out[t];
  const int n0 = blockIdx.y * 64;
  const int p0 = pl.seg_req[t], p1 = pl.seg_req[t + 1];
  if (p0 == p1 || n0 >= n_out) return;
  const float* Wt = (const float*)(HID ? h.W1[t] : h.W[t]);
  const float* bt = HID ? (h.b1 ? (const float*)h.b1[t] : nullptr) : (h.b ? (const float*)h.b[t] : nullptr);
  const bool from_hid = !HID && mlp;
  const int K = from_hid ? h.hidden : d;
  const float* in = from_hid ? hid : pooled;
  for (int e = threadIdx.x; e < (p1 - p0) * 64; e += 256) {
    const int p = p0 + e / 64, n = n0 + e % 64;
    if (n >= n_out) continue;
    float s = bt ? bt[n] : 0.f;
    for (int k = 0; k < K; ++k) s += in[(int64_t)p * K + k] * Wt[(int64_t)n * K + k];
    if (HID) {
      hid[(int64_t)p * h.hidden + n] =
          h.act == VFM_ACT_RELU ? fmaxf(s, 0.f) : 0.5f * s * (1.f + erff(s * 0.70710678118654752440f));
    } else {
      const int req = pl.order[p];
      if (n >= min(n_out, pl.out_off[req + 1] - pl.out_off[req])) continue;
      out[pl.out_off[req] + n] = s;
    }
  }
}


// ---------------------------------------------------------------------------
// Greedy token selection: one block per request (original order), each
// thread scans a strided share of the request's outputs, then the wave and
// the block reduce (value, index) pairs.
// ---------------------------------------------------------------------------
__device__ inline bool greedy_better(float v, int i, float bv, int bi) {
  if (i < 0) return false;
  if (bi < 0) return true;
  return v > bv || (v == bv && i < bi);
}

__global__ __launch_bounds__(256) void greedy_kernel(Plan pl, const float* __restrict__ out,
                                                     int32_t* __restrict__ ids) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int i = blockIdx.x;
  const int o0 = pl.out_off[i], n = pl.out_off[i + 1] - o0;
  float bv = 0.f;
  int bi = -1;
  for (int j = threadIdx.x; j < n; j += 256) {
    const float v = out[o0 + j];
    if (v == v && greedy_better(v, j, bv, bi)) { bv = v; bi = j; }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float ov = __shfl_xor(bv, off, 64);
    const int oi = __shfl_xor(bi, off, 64);
    if (greedy_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) { sv[wave] = bv; si[wave] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (greedy_better(sv[w], si[w], bv, bi)) { bv = sv[w]; bi = si[w]; }
    ids[i] = bi;
  }
}

}  // namespace

hipError_t launch_lora_shrink(int dtype, const Plan& pl, const ShrinkArgs& a, hipStream_t s) {
  if (pl.n_rtiles == 0 || a.n_proj == 0) return hipSuccess;
  if (dtype == VFM_BF16) {
    // the plan's 64-row tiles while one round of blocks holds them, else
    // 96-row tiles (a bound on their count; blocks past the last one leave)
    const bool big = pl.n_rtiles > 256;
    const dim3 grid(big ? (pl.T + 95) / 96 + std::min(pl.n_tasks, pl.n_req) : pl.n_rtiles);
    // sub-tiles the table's ranks need: 1 (rank <= 16), 2 (<= 32) or 4
    const int ns = a.nsub <= 1 ? 1 : (a.nsub == 2 ? 2 : 4);
#define SHR(NP_, NS_)                                                                              \
  do {                                                                                             \
    if (big) hipLaunchKernelGGL((shrink_bf16_kernel<NP_, NS_, 6>), grid, dim3(384), 0, s, pl, a); \
    else hipLaunchKernelGGL((shrink_bf16_kernel<NP_, NS_, 4>), grid, dim3(256), 0, s, pl, a);     \
  } while (0)
#define SHR_NP(NS_) do { if (a.n_proj == 1) SHR(1, NS_); else if (a.n_proj == 2) SHR(2, NS_); else SHR(3, NS_); } while (0)
    if (ns == 1) SHR_NP(1);
    else if (ns == 2) SHR_NP(2);
    else SHR_NP(4);
#undef SHR_NP
#undef SHR
  } else if (a.K % 4 == 0) {
    dim3 grid(4 * pl.n_rtiles, a.n_proj);
    hipLaunchKernelGGL(shrink_f32_stream_kernel, grid, dim3(256), 0, s, pl, a);
  } else {
    dim3 grid(pl.n_rtiles, a.n_proj);
    hipLaunchKernelGGL(shrink_f32_kernel, grid, dim3(256), 0, s, pl, a);
  }
  return hipGetLastError();
}

hipError_t launch_lora_expand(int dtype, const Plan& pl, const ExpandArgs& a, hipStream_t s) {
  if (pl.n_rtiles == 0) return hipSuccess;
  dim3 grid(pl.n_rtiles, (a.N + 63) / 64);
  if (dtype == VFM_BF16) hipLaunchKernelGGL(expand_bf16_kernel, grid, dim3(256), 0, s, pl, a);
  else hipLaunchKernelGGL(expand_f32_kernel, grid, dim3(256), 0, s, pl, a);
  return hipGetLastError();
}

// The pooled rows sit at the start of the head workspace; the MLP heads'
// hidden rows follow at the next 256-byte boundary ([n_req, hidden]).
hipError_t launch_heads(int dtype, const Plan& pl, const void* pooled, int d,
                        const vfm_head_table& h, float* out, hipStream_t s) {
  const size_t es = dtype == VFM_BF16 ? 2 : 4;
  char* hid = (char*)pooled + (((size_t)pl.n_req * d * es + 255) & ~(size_t)255);
  if (h.W1 && h.hidden > 0) {
    dim3 g1(h.n_tasks, (h.hidden + 63) / 64);
    if (dtype == VFM_BF16)
      hipLaunchKernelGGL((heads_bf16_kernel<true>), g1, dim3(256), 0, s, pl, (const bf16*)pooled, d, h,
                         (bf16*)hid, out);
    else
      hipLaunchKernelGGL((heads_f32_kernel<true>), g1, dim3(256), 0, s, pl, (const float*)pooled, d, h,
                         (float*)hid, out);
  }
  dim3 grid(h.n_tasks, (h.max_out + 63) / 64);
  if (grid.y == 0) return hipGetLastError();
  if (dtype == VFM_BF16)
    hipLaunchKernelGGL((heads_bf16_kernel<false>), grid, dim3(256), 0, s, pl, (const bf16*)pooled, d, h,
                       (bf16*)hid, out);
  else
    hipLaunchKernelGGL((heads_f32_kernel<false>), grid, dim3(256), 0, s, pl, (const float*)pooled, d, h,
                       (float*)hid, out);
  return hipGetLastError();
}

hipError_t launch_greedy(const Plan& pl, const float* out, int32_t* ids, hipStream_t s) {
  hipLaunchKernelGGL(greedy_kernel, dim3(pl.n_req), dim3(256), 0, s, pl, out, ids);
  return hipGetLastError();
}
