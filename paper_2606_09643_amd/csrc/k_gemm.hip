// Shared projections (a3, a7, a9, a10): ONE GEMM over every row of the mixed
// batch, C[m, n] = sum_k X[m, k] W[n, k], with the per-task LoRA expand fused
// in as extra MFMA steps and the bias / activation / residual fused into the
// epilogue.
//
// The paper batches all requests through the shared backbone and then adds
// each adapter's difference on its own requests (Section 4.2, adapter
// handling; Fig. 5 (c)).  Here the difference is not a second pass over the
// output: after the K loop, a tile that holds rows of tasks t0..t1 (rows are
// sorted by task, so a tile spans a contiguous task range) runs, per task,
// ceil(r_t / 32) more MFMA steps with A-operand B_t (the task's expand factor,
// read straight from its device pointer) and B-operand U (the per-row shrink
// output s_t x A_t^T), masked to that task's rows.  The sum is exactly
// x W^T + s_t (x A_t^T) B_t^T per row.
//
// bf16 path (gfx950): v_mfma_f32_16x16x32_bf16, 128x128x64 block tile,
// 4 waves of 64x64, LDS double buffer with an XOR swizzle so that both the
// 16-byte fragment reads and the row writes are bank-conflict free, global
// loads for tile k+1 in flight during the MFMAs of tile k.  The weight tile
// feeds the MFMA A slot and the activation tile the B slot, so each lane ends
// up with 4 consecutive output columns of one row: epilogue stores are 8-byte
// (bf16) or 16-byte (fp32) vectors.
//
// fp32 path: a plain LDS-tiled FMA GEMM with the same epilogues (the tiny
// fp32 encoder workload only needs exactness, not speed).
#include <type_traits>

#include "vfm_internal.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 64;

// LDS chunk swizzle of a [rows][64 bf16] tile (128-byte rows, eight 16-byte
// chunks): logical chunk kc of row r lives at physical chunk kc ^ ((r >> 1) & 7).
// Measured on gfx950 with the LDS bank-conflict counter: zero conflicts for
// the ds_read_b128 fragment reads of both the 16x16 and the 32x32 MFMA
// operand layouts (rows r..r+15 at one logical chunk).
__device__ __forceinline__ int swz_bits(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swz(int row, int kc) { return kc ^ swz_bits(row); }

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.f + erff(v * 0.70710678118654752440f));
}
__device__ __forceinline__ float silu_exact(float v) { return v / (1.f + expf(-v)); }  // fp32 outputs

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;

// Fused per-task LoRA expand for one wave's FM x FN fragment grid (shared by
// both bf16 kernels).  wrow0 / wcol0: the wave's first row / first B-tile row.
template <int FM, int FN, bool SWIGLU>
__device__ __forceinline__ void lora_expand_frags(const GemmArgs& a, int m0, int BMrows, int wrow0,
                                                  int n0, int wcol0, int lane,
                                                  f32x4 (&acc)[FM][FN]) {
  const GemmLora& L = a.lora;
  const bf16* U = (const bf16*)L.U;
  const int mlast = min(m0 + BMrows, a.M) - 1;
  const int t0 = L.row_task[m0], t1 = L.row_task[mlast];
  for (int t = t0; t <= t1; ++t) {
    const int r = min(L.rank[t], L.max_rank) & ~7;
    if (r <= 0) continue;
    const int s0 = L.seg_row[t], s1 = L.seg_row[t + 1];
    if (s1 <= wrow0 || s0 >= wrow0 + FM * 16) continue;
    for (int kk = 0; kk < r; kk += 32) {
      const int kof = kk + 8 * (lane >> 4);
      const bool kin = kof < r;
      bf16x8 xf[FM];
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) xf[mi] = bf16x8{};
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        int slot, nrow, nlim;
        if (SWIGLU) {
          const int sub = wcol0 / 16 + ni;
          slot = sub & 1;
          const int jb = n0 + (sub >> 1) * 16;
          if (jb >= a.N) continue;
          nrow = jb + (lane & 15);
          nlim = a.N;
        } else {
          const int nb = n0 + wcol0 + ni * 16;
          if (nb >= a.N) continue;
          slot = nb / L.slot_width;
          nrow = nb - slot * L.slot_width + (lane & 15);
          nlim = L.slot_width;
        }
        if (L.B[slot] == nullptr) continue;
        const bf16* Bt = (const bf16*)L.B[slot][t];
        bf16x8 wf = {};
        if (kin && nrow < nlim) wf = *reinterpret_cast<const bf16x8*>(Bt + (int64_t)nrow * r + kof);
#pragma unroll
        for (int mi = 0; mi < FM; ++mi) {
          const int m = wrow0 + mi * 16 + (lane & 15);
          bf16x8 x = {};
          if (m >= s0 && m < s1 && m < a.M)
            x = *reinterpret_cast<const bf16x8*>(U + (int64_t)m * L.ldu + L.ucol[slot] + kof);
          acc[mi][ni] = mfma16(wf, x, acc[mi][ni]);
        }
      }
    }
  }
}

// Epilogue for one wave's FM x FN fragment grid; lane holds 4 consecutive
// output columns of one row per fragment.  Bias is read once per column
// group and the residual loads of a row group are issued together, so the
// global-memory latency is paid FM times, not FM x FN times.
template <int EPI, bool SWIGLU, int FM, int FN>
__device__ __forceinline__ void epilogue_frags(const GemmArgs& a, int wrow0, int n0, int wcol0,
                                               int lane, const f32x4 (&acc)[FM][FN]) {
  if (SWIGLU) {
#pragma unroll
    for (int mi = 0; mi < FM; ++mi) {
      const int m = wrow0 + mi * 16 + (lane & 15);
      if (m >= a.M) continue;
#pragma unroll
      for (int ni = 0; ni < FN; ni += 2) {
        const int sub = wcol0 / 16 + ni;
        const int j = n0 + (sub >> 1) * 16 + 4 * (lane >> 4);
        if (j >= a.N) continue;
        bf16x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = (bf16)(silu_fast(acc[mi][ni][r]) * acc[mi][ni + 1][r]);
        *reinterpret_cast<bf16x4*>((bf16*)a.out + (int64_t)m * a.ldo + j) = o;
      }
    }
    return;
  }
  const bf16* bias = (const bf16*)a.bias;
  f32x4 bv[FN];
#pragma unroll
  for (int ni = 0; ni < FN; ++ni) {
    bv[ni] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int n = n0 + wcol0 + ni * 16 + 4 * (lane >> 4);
    if (bias && n < a.N) {
      const bf16x4 bb = *reinterpret_cast<const bf16x4*>(bias + n);
#pragma unroll
      for (int r = 0; r < 4; ++r) bv[ni][r] = (float)bb[r];
    }
  }
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int m = wrow0 + mi * 16 + (lane & 15);
    if (m >= a.M) continue;
    if (EPI == EPI_RESID) {
      float* row = (float*)a.out + (int64_t)m * a.ldo;
      float4 old[FN];
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        const int n = n0 + wcol0 + ni * 16 + 4 * (lane >> 4);
        old[ni] = n < a.N ? *reinterpret_cast<const float4*>(row + n) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        const int n = n0 + wcol0 + ni * 16 + 4 * (lane >> 4);
        if (n >= a.N) continue;
        float4 o = old[ni];
        o.x += acc[mi][ni][0] + bv[ni][0];
        o.y += acc[mi][ni][1] + bv[ni][1];
        o.z += acc[mi][ni][2] + bv[ni][2];
        o.w += acc[mi][ni][3] + bv[ni][3];
        *reinterpret_cast<float4*>(row + n) = o;
      }
    } else {
      bf16* row = (bf16*)a.out + (int64_t)m * a.ldo;
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        const int n = n0 + wcol0 + ni * 16 + 4 * (lane >> 4);
        if (n >= a.N) continue;
        bf16x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = acc[mi][ni][r] + bv[ni][r];
          o[r] = (bf16)(EPI == EPI_GELU ? gelu_fast(v) : v);
        }
        *reinterpret_cast<bf16x4*>(row + n) = o;
      }
    }
  }
}

// Epilogue of the large-M kernel through LDS.  The MFMA fragments leave each
// lane with 4 consecutive columns of 16 different rows, so direct stores are
// 16 row pieces of 32 B (bf16) or 64 B (fp32) per instruction.  Here the
// finished values (bias, activation applied) go into the idle operand LDS as
// a row-major tile first, and the block then writes whole rows, 16 B per lane
// with consecutive lanes on consecutive addresses.  16-byte chunk q of tile
// row r sits at chunk q ^ (r & S), S + 1 the largest power of two (at most 8)
// dividing the row's chunk count, which spreads the fragment writes of
// consecutive rows over distinct banks.  The fp32 residual tile (4 B per
// value) is done in two halves of rows.
template <int QR>
__device__ __forceinline__ int lds_chunk(int r, int q) {
  constexpr int LOW = QR & -QR, S = (LOW < 8 ? LOW : 8) - 1;
  return q ^ (r & S);
}

template <int EPI, bool SWIGLU, int BMT, int BNT, int FM, int FN>
__device__ __forceinline__ void epilogue_lds(const GemmArgs& a, char* lds, int m0, int n0, int wm, int wn,
                                             int lane, int tid, const f32x4 (&acc)[FM][FN]) {
  constexpr int NTH = 512, TM = BMT / 4, TN = BNT / 2;
  constexpr int NC = SWIGLU ? BNT / 2 : BNT;        // output columns of the tile
  const int g = lane >> 4;
  __syncthreads();                                  // every wave is done with the operand stages
  if (EPI != EPI_RESID) {
    constexpr int QR = NC / 8;                      // 16-byte chunks per row (bf16)
    static_assert(QR % 4 == 0, "row chunks");
    static_assert(BMT * NC * 2 <= 2 * (BMT + BNT) * BK * 2, "tile fits the operand LDS");
    bf16* T = reinterpret_cast<bf16*>(lds);
    if (SWIGLU) {
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) {
        const int r = wm * TM + mi * 16 + (lane & 15);
#pragma unroll
        for (int ni = 0; ni < FN; ni += 2) {
          const int sub = wn * TN / 16 + ni;
          const int j = (sub >> 1) * 16 + 4 * g;     // tile column of the lane's 4 values
          bf16x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (bf16)(silu_fast(acc[mi][ni][e]) * acc[mi][ni + 1][e]);
          *reinterpret_cast<bf16x4*>(T + r * NC + lds_chunk<QR>(r, j >> 3) * 8 + (j & 4)) = o;
        }
      }
    } else {
      const bf16* bias = (const bf16*)a.bias;
      f32x4 bv[FN];
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        bv[ni] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int j = wn * TN + ni * 16 + 4 * g;
        if (bias && n0 + j < a.N) {
          const bf16x4 bb = *reinterpret_cast<const bf16x4*>(bias + n0 + j);
#pragma unroll
          for (int e = 0; e < 4; ++e) bv[ni][e] = (float)bb[e];
        }
      }
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) {
        const int r = wm * TM + mi * 16 + (lane & 15);
        bf16* row = T + r * NC + (g & 1) * 4;
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) {
          const int q = (wn * TN + ni * 16) / 8 + (g >> 1);   // 16-byte chunk of the lane's 4 values
          bf16x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float v = acc[mi][ni][e] + bv[ni][e];
            o[e] = (bf16)(EPI == EPI_GELU ? gelu_fast(v) : v);
          }
          *reinterpret_cast<bf16x4*>(row + lds_chunk<QR>(r, q) * 8) = o;
        }
      }
    }
    __syncthreads();
    bf16* out = (bf16*)a.out;
    if (EPI == EPI_STORE && !SWIGLU && a.rope.on && n0 < 2 * a.rope.d) {   // block-uniform
      // Rotary embedding of the q / k columns on the staged rows (the tile
      // holds whole heads): a thread takes 8 columns i .. i + 7 of a head's
      // first half and their partners i + head_dim / 2, rotates both in
      // fp32 and stores both.  The angle pos * theta^(-2i / head_dim), in
      // revolutions reduced to [0, 1), feeds the hardware sine and cosine.
      const int hc = a.rope.head_dim / 8;            // 16-byte chunks per head
      const int hh = hc / 2;
      const float l2t = a.rope.log2_theta, inv_hd = 2.0f / (float)a.rope.head_dim;
#pragma unroll 2
      for (int e = tid; e < BMT * (QR / 2); e += NTH) {
        const int r = e / (QR / 2), qq = e % (QR / 2);
        const int q1 = (qq / hh) * hc + qq % hh, q2 = q1 + hh;
        const int m = m0 + r;
        const bf16x8 v1 = *reinterpret_cast<const bf16x8*>(T + r * NC + lds_chunk<QR>(r, q1) * 8);
        const bf16x8 v2 = *reinterpret_cast<const bf16x8*>(T + r * NC + lds_chunk<QR>(r, q2) * 8);
        if (m >= a.M) continue;
        const float pf = (float)a.rope.pos[m];
        const int i0 = (qq % hh) * 8;                // frequency index of the first column
        bf16x8 o1, o2;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float x = pf * (exp2f(-(float)(i0 + j) * inv_hd * l2t) * 0.15915494309189535f);
          const float fr = x - floorf(x);
          const float cs = __builtin_amdgcn_cosf(fr), sn = __builtin_amdgcn_sinf(fr);
          const float x1 = (float)v1[j], x2 = (float)v2[j];
          o1[j] = (bf16)(x1 * cs - x2 * sn);
          o2[j] = (bf16)(x2 * cs + x1 * sn);
        }
        bf16* orow = out + (int64_t)m * a.ldo + n0;
        *reinterpret_cast<bf16x8*>(orow + q1 * 8) = o1;
        *reinterpret_cast<bf16x8*>(orow + q2 * 8) = o2;
      }
      return;
    }
#pragma unroll 4
    for (int e = tid; e < BMT * QR; e += NTH) {
      const int r = e / QR, q = e % QR;
      const int m = m0 + r, n = n0 + q * 8;
      const bf16x8 v = *reinterpret_cast<const bf16x8*>(T + r * NC + lds_chunk<QR>(r, q) * 8);
      if (m < a.M && n < a.N) *reinterpret_cast<bf16x8*>(out + (int64_t)m * a.ldo + n) = v;
    }
    return;
  }
  // fp32 residual: x[m, n] += acc + bias, rows of each half staged as fp32
  constexpr int HR = BMT / 2;                       // rows per half
  constexpr int QR = NC / 4;                        // 16-byte chunks per row (fp32)
  static_assert(QR % 4 == 0, "row chunks");
  static_assert(HR * NC * 4 <= 2 * (BMT + BNT) * BK * 2, "half tile fits the operand LDS");
  float* T = reinterpret_cast<float*>(lds);
  const bf16* bias = (const bf16*)a.bias;
  float* x = (float*)a.out;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if ((wm >> 1) == half) {                        // waves wm = 2 half, 2 half + 1 own these rows
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        const int j = wn * TN + ni * 16 + 4 * g;
        float bv[4] = {0.f, 0.f, 0.f, 0.f};
        if (bias && n0 + j < a.N) {
          const bf16x4 bb = *reinterpret_cast<const bf16x4*>(bias + n0 + j);
#pragma unroll
          for (int e = 0; e < 4; ++e) bv[e] = (float)bb[e];
        }
#pragma unroll
        for (int mi = 0; mi < FM; ++mi) {
          const int r = (wm & 1) * TM + mi * 16 + (lane & 15);   // row within the half
          const float4 o = make_float4(acc[mi][ni][0] + bv[0], acc[mi][ni][1] + bv[1],
                                       acc[mi][ni][2] + bv[2], acc[mi][ni][3] + bv[3]);
          *reinterpret_cast<float4*>(T + r * NC + lds_chunk<QR>(r, j >> 2) * 4) = o;
        }
      }
    }
    __syncthreads();
#pragma unroll 4
    for (int e = tid; e < HR * QR; e += NTH) {
      const int r = e / QR, q = e % QR;
      const int m = m0 + half * HR + r, n = n0 + q * 4;
      if (m < a.M && n < a.N) {
        const float4 v = *reinterpret_cast<const float4*>(T + r * NC + lds_chunk<QR>(r, q) * 4);
        float4* dst = reinterpret_cast<float4*>(x + (int64_t)m * a.ldo + n);
        float4 o = *dst;
        o.x += v.x; o.y += v.y; o.z += v.z; o.w += v.w;
        *dst = o;
      }
    }
    if (half == 0) __syncthreads();                 // the second half reuses the buffer
  }
}

// ---------------------------------------------------------------------------
// Large-M bf16 GEMM: BMT x BNT x 64 block tile (256 rows, 128 / 192 / 256
// columns), 8 waves (4 along M x 2 along N) of (BMT/4) x (BNT/2), operands
// streamed global -> LDS with global_load_lds_dwordx4 (no staging registers),
// two LDS stages (up to 128 KB), and an XCD-aware tile order: consecutive
// block ids land on different XCDs (each with its own L2), so block b takes
// logical tile (b % 8) * per + b / 8 and logical tiles run in groups of LGM
// row-tiles sweeping all column tiles, keeping each XCD's X rows and W
// columns resident in its L2.  The launcher picks the tile shape per GEMM
// so that the last round of tiles fills the 256 CUs as far as possible.
//
// The per-task LoRA expand runs as extra 64-wide K steps of the same
// pipeline: for the tasks t with rows in the tile, the A tile holds the
// shrink outputs U[m, slot cols] of t's rows (rows of other tasks zero) and
// the B tile holds B_t[n, :r_t] (zero past the rank); with ranks <= 16 up to
// four tasks share a step, each in its own 16 columns (SwiGLU: two, 16 gate
// and 16 up columns each).  The MFMA loop cannot tell these steps from the
// backbone's.
// ---------------------------------------------------------------------------
constexpr int LGM = 4;


template <int EPI, bool SWIGLU, int BMT, int BNT, bool PACK>
__global__ __launch_bounds__(512, 1) void gemm_bf16_large_kernel(GemmArgs a) {
  constexpr int NW = 8, NTH = 512, WN = 2, TM = BMT / 4, TN = BNT / 2, FM = TM / 16, FN = TN / 16;
  constexpr int ACH = BMT * 8 / NTH, BCH = BNT * 8 / NTH;  // 16-byte chunks per lane and stage
  constexpr int SA = BMT * BK, SB = BNT * BK;
  static_assert(BMT % 64 == 0 && BNT % 64 == 0 && FN % 2 == 0, "tile shape");
  constexpr int RSTEP = NTH / 8;                             // 64 rows per chunk step
  __shared__ __attribute__((aligned(16))) bf16 smem[2 * (SA + SB)];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  constexpr int NTILE = SWIGLU ? BNT / 2 : BNT;  // output columns per block
  const int MT = (a.m_hi - a.m_lo + BMT - 1) / BMT, NTn = (a.N + NTILE - 1) / NTILE, ntiles = MT * NTn;
  const int per = gridDim.x / 8;
  const int Lid = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (Lid >= ntiles) return;
  int tm, tn;
  {
    const int gsz = LGM * NTn;
    const int g = Lid / gsz, r = Lid % gsz;
    const int fm = g * LGM;
    const int gm = min(MT - fm, LGM);
    tm = fm + r % gm;
    tn = r / gm;
  }
  const int m0 = a.m_lo + tm * BMT, n0 = tn * NTILE;
  const bf16* X = (const bf16*)a.X;
  const GemmLora& L = a.lora;

  // Each wave fills whole 1 KB LDS slots (8 rows x 128 B); lane `lane` of
  // chunk i writes LDS row (i*NW + wave)*8 + lane/8, physical 16-byte chunk
  // lane%8, so it loads the logical chunk that the swizzle maps there.
  const int row0 = wave * 8 + (lane >> 3);
  const int kc0 = (lane & 7) ^ swz_bits(row0);  // same for row0 + i * RSTEP
  // element offsets (32-bit: the launcher keeps M * ldx and N * K below 2^31)
  // of each chunk's row, to keep the 64-bit pointer pairs out of registers
  int xoff[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) xoff[i] = min(m0 + row0 + i * RSTEP, a.M - 1) * a.ldx + kc0 * 8;
  int woff[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int row = row0 + i * RSTEP;
    int wrow;
    if (SWIGLU) {
      const int sub = row >> 4;
      wrow = n0 + (sub >> 1) * 16 + (row & 15);
    } else {
      wrow = n0 + row;
    }
    woff[i] = min(wrow, a.N - 1) * a.K + kc0 * 8;
  }
  // SwiGLU: 16-row groups of the B tile alternate gate (W) and up (W2) rows
  auto wbase = [&](int i) -> const bf16* {
    if (SWIGLU && (((row0 + i * RSTEP) >> 4) & 1)) return (const bf16*)a.W2;
    return (const bf16*)a.W;
  };

  // LoRA steps.  Rows are sorted by task, so the tile's rows form runs of
  // one task each.  The task ids of the tile's rows arrive with the first
  // operand DMA (RPL per lane); ballots of the rows that start a run then
  // list the runs, so a task without rows in the tile (an id absent from the
  // batch included) costs no step.  A LoRA step is a 64-column K step whose
  // A tile is U (the slot's columns; rows of other runs zero) and whose B
  // tile is B_t (zero past the rank).  Without PACK a step serves one run:
  // ranks <= 32 fill its first 32 columns (a half step; SwiGLU: gate in the
  // low 32, up in the high 32), a SwiGLU run of a larger rank takes two
  // steps (gate, then up).  With PACK (every rank <= 16) the step's columns
  // are cut into P slots, one run each (16 columns; SwiGLU: 16 gate then 16
  // up), so a tile with many small runs (a few rows each of many tasks)
  // needs a quarter (a half) of the steps.  Every product a row meets
  // outside its own slot has a zero operand, so its sum does not depend on
  // which runs share its step.  A lane's 16-byte chunk of a step row is
  // fixed for the tile, and so is its slot.  A group's task ids come from
  // the tile's row tasks (registers); each lane reads its slot's rank and B
  // pointer from the small per-task tables (cache hits after the first).
  const int nk = a.K / BK;
  constexpr int RPL = BMT / 64;                    // tile rows per lane
  static_assert(BMT % 64 == 0, "rows per lane");
  const int parts = (SWIGLU && L.max_rank > 32) ? 2 : 1;
  // chunks (8 columns) per projection of a slot, chunks per slot, slots per step
  const int hc = PACK ? 2 : L.max_rank > 32 ? 8 : 4;
  const int cwc = (SWIGLU && parts == 1) ? 2 * hc : hc;
  constexpr int P = PACK ? (SWIGLU ? 2 : 4) : 1;
  const int slot = PACK ? kc0 / (SWIGLU ? 4 : 2) : 0;     // this lane's slot
  const int q = PACK ? kc0 % (SWIGLU ? 4 : 2) : kc0;      // and its chunk within the slot
  bool live = false;
  if (L.enabled) {
    if (SWIGLU) live = L.B[0] != nullptr || L.B[1] != nullptr;
    else live = L.B[min(n0 / L.slot_width, 2)] != nullptr;
  }
  const int lslot = SWIGLU ? 0 : min(n0 / L.slot_width, 2);
  int rt[RPL];                                     // task of tile row RPL * lane + j
#pragma unroll
  for (int j = 0; j < RPL; ++j) rt[j] = live ? L.row_task[min(m0 + RPL * lane + j, a.M - 1)] : 0;
  uint64_t rstart[RPL];                            // bit l of rstart[j]: row RPL*l + j starts a run
  int nlora = 0, nsteps = nk;
  auto first_start_ge = [&](int r) -> int {        // first run start at tile row >= r, else BMT
    int best = BMT;
#pragma unroll
    for (int j = 0; j < RPL; ++j) {
      const int lmin = r <= j ? 0 : (r - j + RPL - 1) / RPL;
      if (lmin < 64) {
        const uint64_t m = rstart[j] & (~0ull << lmin);
        if (m) best = min(best, RPL * (int)__builtin_ctzll(m) + j);
      }
    }
    return best;
  };
  auto task_at = [&](int r) -> int {               // task of tile row r (wave-uniform r)
    int t = __builtin_amdgcn_readlane(rt[0], r / RPL);
#pragma unroll
    for (int j = 1; j < RPL; ++j)
      if (r % RPL == j) t = __builtin_amdgcn_readlane(rt[j], r / RPL);
    return t;
  };
  // The current step's group (wave-uniform): the tile rows where it starts
  // and where the next one starts; read when the group's first step is
  // issued (a SwiGLU group of a rank above 32 takes two steps).
  int g_start = 0, g_end = 0;
  int cs = 0, ce = 0, cr = 0;                      // this lane's run: tile rows [cs, ce), rank
  const bf16* cb = nullptr;                        // and B pointer
  bool half_next = false;                          // the issued step fills only its first 32 columns
  auto load_step = [&](int part) {
    const int start = part == 0 ? g_end : g_start;
    int b[P + 1];
    b[0] = start;
#pragma unroll
    for (int u = 1; u <= P; ++u) b[u] = b[u - 1] < BMT ? first_start_ge(b[u - 1] + 1) : BMT;
    int used = 0, mt = -1;
    cs = ce = BMT;
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const bool has = b[u] < BMT;
      const int t = has ? task_at(b[u]) : -1;
      used += has ? cwc : 0;
      if (u == slot) { cs = b[u]; ce = b[u + 1]; mt = t; }
    }
    g_start = start;
    g_end = b[P];
    half_next = used <= 4;
    // the lane's projection: its slot's gate or up half (SwiGLU), else the block's
    const int proj = SWIGLU ? (parts == 2 ? part : (q >= hc ? 1 : 0)) : lslot;
    const void* const* tab = proj == 0 ? L.B[0] : proj == 1 ? L.B[1] : L.B[2];
    cr = 0;
    cb = nullptr;
    if (mt >= 0) {
      cr = min(L.rank[mt], L.max_rank) & ~7;
      if (tab != nullptr) cb = (const bf16*)tab[mt];
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int mi = 0; mi < FM; ++mi)
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto issue_bb = [&](int e) {
    bf16* As = smem + (e & 1) * (SA + SB);
    bf16* Bs = As + SA;
    const int k0 = e * BK;
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      __builtin_amdgcn_global_load_lds((gptr_t)(X + xoff[i] + k0), (lptr_t)(As + (i * NW + wave) * 512), 16, 0, 0);
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      __builtin_amdgcn_global_load_lds((gptr_t)(wbase(i) + woff[i] + k0), (lptr_t)(Bs + (i * NW + wave) * 512), 16,
                                       0, 0);
  };
  // A LoRA-step chunk: lanes with data DMA it, the others write zeros into
  // their own 16-byte LDS slot (a shared zero page read by every CU would
  // funnel those loads into one L2 line).  The step's wait covers both.
  auto dma_or_zero = [&](bool on, const bf16* src, bf16* dst) {
    if (on) __builtin_amdgcn_global_load_lds((gptr_t)src, (lptr_t)dst, 16, 0, 0);
    else *reinterpret_cast<bf16x8*>(dst + lane * 8) = bf16x8{};
  };
  auto issue = [&](int e) {
    bf16* As = smem + (e & 1) * (SA + SB);
    bf16* Bs = As + SA;
    if (e < nk) {
      const int k0 = e * BK;
#pragma unroll
      for (int i = 0; i < ACH; ++i)
        __builtin_amdgcn_global_load_lds((gptr_t)(X + xoff[i] + k0), (lptr_t)(As + (i * NW + wave) * 512), 16, 0, 0);
#pragma unroll
      for (int i = 0; i < BCH; ++i)
        __builtin_amdgcn_global_load_lds((gptr_t)(wbase(i) + woff[i] + k0), (lptr_t)(Bs + (i * NW + wave) * 512), 16,
                                         0, 0);
      return;
    }
    const int step = e - nk, part = step % parts;
    load_step(part);
    const bf16* U = (const bf16*)L.U;
    // this lane's chunk: projection (SwiGLU: gate or up) and chunk within it
    int proj = 0, qq = q;
    if (SWIGLU) {
      if (parts == 2) proj = part;
      else { proj = q >= hc ? 1 : 0; qq = q - proj * hc; }
    }
    // A: the run's rows of U at the slot's columns.  Only columns the shrink
    // wrote are read (the rest are zeroed in LDS), so stale workspace bytes
    // never meet a zero of B.
    const int ucolA = L.ucol[SWIGLU ? proj : lslot] + qq * 8;
    const bool colA = qq * 8 < (L.max_rank > 32 ? 64 : 32) && (!SWIGLU || (proj ? L.B[1] : L.B[0]) != nullptr);
    // with a half step, columns 32..63 are neither loaded nor read
    const bool skip = half_next && kc0 >= 4;
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int row = row0 + i * RSTEP, m = m0 + row;
      const bool on = colA && row >= cs && row < ce && m < a.M;
      if (!skip) dma_or_zero(on, U + (int64_t)m * L.ldu + ucolA, As + (i * NW + wave) * 512);
    }
    // B: B_t rows of this block's output columns, zero past the rank
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int row = row0 + i * RSTEP;
      const bf16* src = nullptr;
      if (SWIGLU) {
        const int sub = row >> 4, which = sub & 1;
        const int j = n0 + (sub >> 1) * 16 + (row & 15);
        if (which == proj && qq * 8 < cr && j < a.N && cb != nullptr) src = cb + (int64_t)j * cr + qq * 8;
      } else {
        const int nrow = n0 + row - lslot * L.slot_width;
        if (qq * 8 < cr && n0 + row < a.N && nrow < L.slot_width && cb != nullptr)
          src = cb + (int64_t)nrow * cr + qq * 8;
      }
      if (!skip) dma_or_zero(src != nullptr, src, Bs + (i * NW + wave) * 512);
    }
  };
  auto compute = [&](int e, bool first_half_only) {
    const bf16* As = smem + (e & 1) * (SA + SB);
    const bf16* Bs = As + SA;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      if (kk == 1 && first_half_only) break;
      const int kc = kk * 4 + (lane >> 4);
      bf16x8 wf[FN];
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) {
        const int r = wn * TN + ni * 16 + (lane & 15);
        wf[ni] = *reinterpret_cast<const bf16x8*>(Bs + r * BK + swz(r, kc) * 8);
      }
#pragma unroll
      for (int mi = 0; mi < FM; ++mi) {
        const int r = wm * TM + mi * 16 + (lane & 15);
        const bf16x8 xf = *reinterpret_cast<const bf16x8*>(As + r * BK + swz(r, kc) * 8);
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) acc[mi][ni] = mfma16(wf[ni], xf, acc[mi][ni]);
      }
    }
  };

  // Waits are explicit: vmcnt(0) makes this wave's LDS-bound loads land, the
  // raw s_barrier then makes every wave's loads visible.  (A full
  // __syncthreads would add a fence the loop does not need.)
  // The backbone K steps run in a loop of their own (its loads are plain
  // strided tiles), then the LoRA steps; the loop that mixes both kinds of
  // issue costs the backbone loop about a tenth of its speed.
  issue_bb(0);
  __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): step 0 and the tile's row tasks
  __builtin_amdgcn_s_barrier();
  if (live) {
    int prev = __shfl_up(rt[RPL - 1], 1, 64);
    if (lane == 0) prev = -1;
#pragma unroll
    for (int j = 0; j < RPL; ++j) {
      const int before = j == 0 ? prev : rt[j - 1];
      rstart[j] = __ballot(rt[j] != before);
    }
    int nruns = 0;
#pragma unroll
    for (int j = 0; j < RPL; ++j) nruns += __builtin_popcountll(rstart[j]);
    nlora = (nruns + P - 1) / P * parts;
    nsteps = nk + nlora;
  }
  if (nk < 2) __builtin_amdgcn_s_waitcnt(0xF70);   // no backbone step covers them
  for (int e = 0; e + 1 < nk; ++e) {
    issue_bb(e + 1);                   // the other stage: every wave left it at the last barrier
    compute(e, false);
    __builtin_amdgcn_s_waitcnt(0xF70);
    __builtin_amdgcn_s_barrier();
  }
  bool half_cur = false;                           // step e fills only its first 32 columns
  for (int e = nk - 1; e < nsteps; ++e) {
    if (e + 1 < nsteps) issue(e + 1);
    compute(e, e >= nk && half_cur);
    half_cur = half_next;
    __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0): DMA and zero writes done
    __builtin_amdgcn_s_barrier();
  }
  // whole rows through LDS (16 B per lane) for the bf16 outputs and for the
  // fp32 residual of tiles narrower than 256 columns; the 256-column
  // residual tile writes from registers (its staged form spills)
  if (EPI != EPI_RESID || BNT < 256)
    epilogue_lds<EPI, SWIGLU, BMT, BNT, FM, FN>(a, reinterpret_cast<char*>(smem), m0, n0, wm, wn, lane, tid,
                                                 acc);
  else
    epilogue_frags<EPI, SWIGLU, FM, FN>(a, m0 + wm * TM, n0, wn * TN, lane, acc);
}

// ---------------------------------------------------------------------------
// Small-M bf16 GEMM (decode-sized batches): 128x128x64, 4 waves of 64x64,
// register-staged LDS double buffer, more blocks for few rows.
// ---------------------------------------------------------------------------
template <int EPI, bool SWIGLU>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * BK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int NT = SWIGLU ? BN / 2 : BN;  // output columns per block
  const int n_tiles_n = (a.N + NT - 1) / NT;
  const int tn = blockIdx.x % n_tiles_n, tm = blockIdx.x / n_tiles_n;
  const int m0 = tm * BM, n0 = tn * NT;
  const bf16* X = (const bf16*)a.X;
  const bf16* W = (const bf16*)a.W;
  const bf16* W2 = (const bf16*)a.W2;

  const bf16* xsrc[4];
  const bf16* wsrc[4];
  int lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    const int m = min(m0 + row, a.M - 1);
    xsrc[i] = X + (int64_t)m * a.ldx + kc * 8;
    const bf16* wb = W;
    int wrow;
    if (SWIGLU) {
      const int sub = row >> 4;
      wb = (sub & 1) ? W2 : W;
      wrow = min(n0 + (sub >> 1) * 16 + (row & 15), a.N - 1);
    } else {
      wrow = min(n0 + row, a.N - 1);
    }
    wsrc[i] = wb + (int64_t)wrow * a.K + kc * 8;
    lds_off[i] = row * BK + swz(row, kc) * 8;
  }

  bf16x8 xr[4], wr[4];
  f32x4 acc[4][4];
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = a.K / BK;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    xr[i] = *reinterpret_cast<const bf16x8*>(xsrc[i]);
    wr[i] = *reinterpret_cast<const bf16x8*>(wsrc[i]);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<bf16x8*>(&As[0][lds_off[i]]) = xr[i];
    *reinterpret_cast<bf16x8*>(&Bs[0][lds_off[i]]) = wr[i];
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt & 1;
    if (kt + 1 < nk) {
      const int k0 = (kt + 1) * BK;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xr[i] = *reinterpret_cast<const bf16x8*>(xsrc[i] + k0);
        wr[i] = *reinterpret_cast<const bf16x8*>(wsrc[i] + k0);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int kc = kk * 4 + (lane >> 4);
      bf16x8 wf[4], xf[4];
#pragma unroll
      for (int ni = 0; ni < 4; ++ni) {
        const int r = wn * 64 + ni * 16 + (lane & 15);
        wf[ni] = *reinterpret_cast<const bf16x8*>(&Bs[st][r * BK + swz(r, kc) * 8]);
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi) {
        const int r = wm * 64 + mi * 16 + (lane & 15);
        xf[mi] = *reinterpret_cast<const bf16x8*>(&As[st][r * BK + swz(r, kc) * 8]);
      }
#pragma unroll
      for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = mfma16(wf[ni], xf[mi], acc[mi][ni]);
    }
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        *reinterpret_cast<bf16x8*>(&As[st ^ 1][lds_off[i]]) = xr[i];
        *reinterpret_cast<bf16x8*>(&Bs[st ^ 1][lds_off[i]]) = wr[i];
      }
    }
    __syncthreads();
  }

  const int wrow0 = m0 + wm * 64;
  if (a.lora.enabled)
    lora_expand_frags<4, 4, SWIGLU>(a, m0, BM, wrow0, n0, wn * 64, lane, acc);
  epilogue_frags<EPI, SWIGLU, 4, 4>(a, wrow0, n0, wn * 64, lane, acc);
}

// ---------------------------------------------------------------------------
// fp32: LDS-tiled FMA GEMM, 64x64 tile, 4x4 outputs per thread.
// ---------------------------------------------------------------------------
template <int EPI, bool SWIGLU>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  constexpr int TM = 64, TN = 64, TK = 16;
  __shared__ float Xs[TK][TM + 4];
  __shared__ float Ws[TK][TN + 4];
  __shared__ float W2s[SWIGLU ? TK : 1][TN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int n_tiles_n = (a.N + TN - 1) / TN;
  const int tn = blockIdx.x % n_tiles_n, tm = blockIdx.x / n_tiles_n;
  const int m0 = tm * TM, n0 = tn * TN;
  const float* X = (const float*)a.X;
  const float* W = (const float*)a.W;
  const float* W2 = (const float*)a.W2;
  const int lrow = tid >> 2, kq = (tid & 3) * 4;
  const int xm = min(m0 + lrow, a.M - 1), wn_ = min(n0 + lrow, a.N - 1);
  float acc[4][4] = {}, acc2[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += TK) {
    const float4 xv = *reinterpret_cast<const float4*>(X + (int64_t)xm * a.ldx + k0 + kq);
    const float4 wv = *reinterpret_cast<const float4*>(W + (int64_t)wn_ * a.K + k0 + kq);
    Xs[kq + 0][lrow] = xv.x; Xs[kq + 1][lrow] = xv.y; Xs[kq + 2][lrow] = xv.z; Xs[kq + 3][lrow] = xv.w;
    Ws[kq + 0][lrow] = wv.x; Ws[kq + 1][lrow] = wv.y; Ws[kq + 2][lrow] = wv.z; Ws[kq + 3][lrow] = wv.w;
    if (SWIGLU) {
      const float4 w2 = *reinterpret_cast<const float4*>(W2 + (int64_t)wn_ * a.K + k0 + kq);
      W2s[kq + 0][lrow] = w2.x; W2s[kq + 1][lrow] = w2.y; W2s[kq + 2][lrow] = w2.z; W2s[kq + 3][lrow] = w2.w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      float xa[4], wb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) xa[i] = Xs[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wb[j] = Ws[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += xa[i] * wb[j];
      if (SWIGLU) {
#pragma unroll
        for (int j = 0; j < 4; ++j) wb[j] = W2s[k][tx * 4 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc2[i][j] += xa[i] * wb[j];
      }
    }
    __syncthreads();
  }

  if (a.lora.enabled) {
    const GemmLora& L = a.lora;
    const float* U = (const float*)L.U;
    const int mlast = min(m0 + TM, a.M) - 1;
    const int t0 = L.row_task[m0], t1 = L.row_task[mlast];
    for (int t = t0; t <= t1; ++t) {
      const int r = min(L.rank[t], L.max_rank) & ~7;
      if (r <= 0) continue;
      const int s0 = L.seg_row[t], s1 = L.seg_row[t + 1];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m < s0 || m >= s1 || m >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + tx * 4 + j;
          if (n >= a.N) continue;
          const int slot = SWIGLU ? 0 : n / L.slot_width;
          const int nrow = SWIGLU ? n : n - slot * L.slot_width;
          if (L.B[slot] != nullptr) {
            const float* Bt = (const float*)L.B[slot][t];
            const float* u = U + (int64_t)m * L.ldu + L.ucol[slot];
            float s = 0.f;
            for (int q = 0; q < r; ++q) s += u[q] * Bt[(int64_t)nrow * r + q];
            acc[i][j] += s;
          }
          if (SWIGLU && L.B[1] != nullptr) {
            const float* Bt2 = (const float*)L.B[1][t];
            const float* u2 = U + (int64_t)m * L.ldu + L.ucol[1];
            float s2 = 0.f;
            for (int q = 0; q < r; ++q) s2 += u2[q] * Bt2[(int64_t)nrow * r + q];
            acc2[i][j] += s2;
          }
        }
      }
    }
  }

  const float* bias = (const float*)a.bias;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    const int n = n0 + tx * 4;
    if (m >= a.M || n >= a.N) continue;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = acc[i][j] + (bias ? bias[n + j] : 0.f);
      if (SWIGLU) v[j] = silu_exact(acc[i][j]) * acc2[i][j];
      else if (EPI == EPI_GELU) v[j] = gelu_erf(v[j]);
    }
    float* dst = (float*)a.out + (int64_t)m * a.ldo + n;
    if (EPI == EPI_RESID) {
      float4 o = *reinterpret_cast<float4*>(dst);
      o.x += v[0]; o.y += v[1]; o.z += v[2]; o.w += v[3];
      *reinterpret_cast<float4*>(dst) = o;
    } else {
      *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// Tile shapes of the large GEMM for an M x N product.  A launch of R tiles
// costs its rounds of 256 concurrent tiles (one per CU) times the bytes a
// tile moves per K step (BMT + BNT rows of 128 B; the loop is bound by that
// stream).  The candidates are the shapes whose column tiles do not straddle
// a LoRA slot.  Besides one launch of the cheapest shape, the rows may be
// split: whole 256-row tiles of one shape in full rounds, then the remaining
// rows with narrower tiles, so the last, partly filled round costs less.
// Every shape runs the same K steps in the same order, so a row's outputs do
// not depend on which launch or tile shape computes it.
struct LargeShape { int bm, bn; };
constexpr LargeShape kLargeShapes[3] = {{256, 256}, {256, 192}, {256, 128}};
inline bool shape_ok(const LargeShape& c, bool sw, int lora_slot_width, int rope_hd) {
  return !(lora_slot_width > 0 && !sw && lora_slot_width % c.bn) && !(rope_hd > 0 && c.bn % rope_hd);
}
inline double launch_cost(int rows, int N, bool sw, const LargeShape& c) {
  if (rows <= 0) return 0.0;
  const int nt = sw ? c.bn / 2 : c.bn;
  const long tiles = (long)((rows + c.bm - 1) / c.bm) * ((N + nt - 1) / nt);
  const long rounds = (tiles + 255) / 256;
  return (double)rounds * (c.bm + c.bn) * (sw ? 2.0 * nt / c.bn : 1.0);
}
struct LargePlan { LargeShape main, tail; int m1; };   // rows [0, m1) main, [m1, M) tail
inline LargePlan large_plan(int M, int N, bool sw, int lora_slot_width, int rope_hd) {
  LargePlan best = {{0, 0}, {0, 0}, M};
  double best_cost = 0.0;
  for (const LargeShape& c : kLargeShapes) {
    if (!shape_ok(c, sw, lora_slot_width, rope_hd)) continue;
    const double cost = launch_cost(M, N, sw, c);
    if (best.main.bm == 0 || cost < best_cost * 0.97) { best = {c, {0, 0}, M}; best_cost = cost; }
  }
  if (best.main.bm == 0) return best;
  const double single = best_cost;
  const LargeShape mc = best.main;
  const int nt = sw ? mc.bn / 2 : mc.bn;
  const int ntn = (N + nt - 1) / nt, mt = (M + mc.bm - 1) / mc.bm;
  // A last round under a quarter full already runs well below a full
  // round's time (its few tiles do not share L2 and HBM bandwidth): no split
  // (measured: the 7B QKV's 32-tile last round is cheaper than a 256 x 128
  // tail launch).  Otherwise a split must beat the single launch by 1.5%.
  const int last = (int)(((long)mt * ntn) % 256);
  if (last == 0 || last < 64) return best;
  const int full = (int)(((long)mt * ntn) / 256 * 256 / ntn);   // row tiles filling whole rounds
  for (int r1 = full; r1 >= 1 && r1 >= full - 2; --r1) {
    const int m1 = r1 * mc.bm;
    if (m1 >= M) continue;
    for (const LargeShape& t : kLargeShapes) {
      if (!shape_ok(t, sw, lora_slot_width, rope_hd)) continue;
      const double cost = launch_cost(m1, N, sw, mc) + launch_cost(M - m1, N, sw, t);
      if (cost < single * 0.985 && cost < best_cost) { best = {mc, t, m1}; best_cost = cost; }
    }
  }
  return best;
}

template <int EPI, bool SW, int BMT, int BNT>
void launch_large(const GemmArgs& a, hipStream_t s) {
  const int nt = SW ? BNT / 2 : BNT;
  const int ntiles = ((a.m_hi - a.m_lo + BMT - 1) / BMT) * ((a.N + nt - 1) / nt);
  const int grid = (ntiles + 7) / 8 * 8;
  // ranks <= 16 share LoRA steps (up to four runs per step)
  if (a.lora.enabled && a.lora.max_rank <= 16)
    hipLaunchKernelGGL((gemm_bf16_large_kernel<EPI, SW, BMT, BNT, true>), dim3(grid), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL((gemm_bf16_large_kernel<EPI, SW, BMT, BNT, false>), dim3(grid), dim3(512), 0, s, a);
}
template <int EPI, bool SW>
void launch_large_shape(const GemmArgs& a, const LargeShape& sh, hipStream_t s) {
  if (sh.bn == 256) launch_large<EPI, SW, 256, 256>(a, s);
  else if (sh.bn == 192) launch_large<EPI, SW, 256, 192>(a, s);
  else launch_large<EPI, SW, 256, 128>(a, s);
}

template <int EPI, bool SW>
hipError_t launch_one(int dtype, const GemmArgs& a0, hipStream_t s) {
  // the fused rotary embedding needs whole heads in a tile
  const LargePlan pl = large_plan(a0.M, a0.N, SW, a0.lora.enabled ? a0.lora.slot_width : 0,
                                  a0.rope.on ? a0.rope.head_dim : 0);
  const bool fits32 = (int64_t)a0.M * a0.ldx < ((int64_t)1 << 31) && (int64_t)a0.N * a0.K < ((int64_t)1 << 31);
  if (dtype == VFM_BF16 && a0.M >= 1024 && pl.main.bm > 0 && fits32) {
    GemmArgs a = a0;
    a.m_lo = 0;
    a.m_hi = pl.m1;
    launch_large_shape<EPI, SW>(a, pl.main, s);
    if (pl.m1 < a0.M) {
      a.m_lo = pl.m1;
      a.m_hi = a0.M;
      launch_large_shape<EPI, SW>(a, pl.tail, s);
    }
  } else if (a0.rope.on) {
    return hipErrorInvalidValue;   // only the large-tile kernel applies the rotary embedding
  } else if (dtype == VFM_BF16) {
    const GemmArgs& a = a0;
    const int nt = SW ? BN / 2 : BN;
    const int grid = ((a.M + BM - 1) / BM) * ((a.N + nt - 1) / nt);
    hipLaunchKernelGGL((gemm_bf16_kernel<EPI, SW>), dim3(grid), dim3(256), 0, s, a);
  } else {
    const GemmArgs& a = a0;
    const int grid = ((a.M + 63) / 64) * ((a.N + 63) / 64);
    hipLaunchKernelGGL((gemm_f32_kernel<EPI, SW>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  switch (a.epi) {
    case EPI_STORE: return launch_one<EPI_STORE, false>(dtype, a, s);
    case EPI_GELU: return launch_one<EPI_GELU, false>(dtype, a, s);
    case EPI_RESID: return launch_one<EPI_RESID, false>(dtype, a, s);
    case EPI_SWIGLU: return launch_one<EPI_STORE, true>(dtype, a, s);
  }
  return hipErrorInvalidValue;
}
