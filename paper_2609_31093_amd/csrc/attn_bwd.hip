// Backward of the selected sparse attention with the selection held fixed
// (App. B: during backpropagation the selected block indices are constants;
// gradients flow through the attention over the selected entries only).
//
// With z = q.k / sqrt(d) over a row's selected visible tokens, p = softmax(z),
// o = sum p v and the output gradient do:
//   dv_j += p_j do,  dp_j = do.v_j,  D = do.o,  ds_j = p_j (dp_j - D),
//   dq = sum_j ds_j k_j / sqrt(d),  dk_j += ds_j q / sqrt(d).
//
// attn_bwd_prep_kernel: per (row, query head) the forward's log-sum in log2
// units and D = do.o.
// attn_bwd_block_kernel: block-centric, like the forward's block kernel.  A
// workgroup owns a chunk of up to kBwdChunk (row, slot) pairs that selected
// one key block; K (row-major and transposed) and V are staged in LDS once.
// Every 64 (pair, head) columns (16 per wavefront) are one MFMA group:
// S^T = K q^T and dP^T = V do^T on v_mfma_f32_16x16x32_bf16, P = 2^(S - lse),
// dS = P (dP - D); dq^T = K^T dS^T gives each pair's dq partial (bf16, like
// the forward's o partials); P^T, dS^T, q and do of the group go to LDS and
// the four wavefronts then add dV += P^T do and dK += dS^T q for their
// quarter of the head dimension, accumulating over the whole chunk in
// registers.  At the end a chunk writes its dK, dV rows in the problem dtype
// when it is its block's only chunk and the launch covers every row, else
// adds them into fp32 accumulators.
// attn_bwd_dq_kernel: dq of each row = the sum of its slots' partials.
// attn_bwd_blocks_kernel / attn_bwd_finalize_kernel: the accumulators (of the
// blocks with several chunks, or all of them) to the problem dtype, and zero
// rows for keys nothing selected.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace pisa {

typedef __bf16 bf16x8b2 __attribute__((ext_vector_type(8)));
typedef float f32x4b2 __attribute__((ext_vector_type(4)));

constexpr int kBwdChunk = 2048;  // pairs per workgroup of the block kernel
constexpr int kBwdCols = 64;     // (pair, head) columns per MFMA group

struct AttnBwdArgs {
  int H, Hkv, G, Nq, N, C, K, causal, M1;
  int row0, nrows;  // row chunk of this launch
  float qscale2;    // log2(e) / sqrt(d)
  float rscale;     // 1 / sqrt(d)
  int Nkv;          // rows per (batch, KV head) in k, v, dk, dv
  // one launch covers every row: a block whose pairs fit one chunk writes
  // its dK, dV rows directly in the problem dtype
  int direct = 0;
};

__device__ __forceinline__ bf16x8b2 u4_bf16x8b2(uint4 r) { return __builtin_bit_cast(bf16x8b2, r); }

// DPL (4 or 8) floats to bf16 (round to nearest even) at p.
template <int DPL>
__device__ __forceinline__ void store_bf16_part(uint16_t* p, const float (&x)[DPL]) {
  if constexpr (DPL == 8) {
    *reinterpret_cast<uint4*>(p) =
        make_uint4(pack2_bf16(x[0], x[1]), pack2_bf16(x[2], x[3]), pack2_bf16(x[4], x[5]), pack2_bf16(x[6], x[7]));
  } else {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack2_bf16(x[0], x[1]), pack2_bf16(x[2], x[3]));
  }
}

// Blocks of 64 keys use a compact LDS layout: every tile unpadded, the
// 16-byte chunks of each row XOR-swizzled, and each wavefront's dq staging
// rows laid over its own P and dS rows, so that (at d = 128) the workgroup
// needs 80 KB and two fit a CU.  Other block sizes keep padded rows.
__host__ __device__ constexpr bool bwd_compact(int C) { return C == 64; }
__host__ __device__ constexpr int bwd_region(int C, int D) { return 2 * 16 * C > 16 * D ? 2 * 16 * C : 16 * D; }
__host__ __device__ constexpr size_t bwd_lds_elems(int C, int D) {
  return bwd_compact(C)
             ? 2 * static_cast<size_t>(C) * D + 2 * static_cast<size_t>(kBwdCols) * D + 4 * static_cast<size_t>(bwd_region(C, D))
             : 2 * static_cast<size_t>(C) * (D + 8) + 2 * static_cast<size_t>(kBwdCols) * (C + 8) +
                   2 * static_cast<size_t>(kBwdCols) * (D + 8) + 4 * 16 * static_cast<size_t>(D + 8);
}

// Chunk swizzles of the compact layout (NCH 16-byte chunks per row): one for
// tiles read 16 consecutive rows at a time (K, V, the dq staging rows), one
// for tiles read by the transposing loads of rows 8 g + j (q, do, P, dS);
// either spreads each read over the banks in the fewest cycles.
template <int NCH>
__device__ __forceinline__ int bwd_swz_rows(int r) {
  return NCH == 16 ? (r & 15) : ((r >> 1) & 7);
}
template <int NCH>
__device__ __forceinline__ int bwd_swz_cols(int r) {
  return NCH == 16 ? ((r & 15) ^ ((r >> 2) & 12)) : 2 * (((r >> 3) + (r >> 1)) & 3);
}

// stat[(b*H + h)*Nq + row] = (lse * log2(e), do . o): 16 lanes per (row, head).
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_prep_kernel(AttnBwdArgs a, const uint16_t* __restrict__ o,
                                                            const uint16_t* __restrict__ dO,
                                                            const float* __restrict__ lse, float2* __restrict__ stat,
                                                            int64_t nrh) {
  constexpr int DPL = D / 16;
  const int sub = threadIdx.x & 15;
  const int64_t rh = static_cast<int64_t>(blockIdx.x) * 16 + (threadIdx.x >> 4);
  if (rh >= nrh) return;
  float x[DPL], y[DPL];
  load_row_part<uint16_t, DPL>(o + rh * D + sub * DPL, x);
  load_row_part<uint16_t, DPL>(dO + rh * D + sub * DPL, y);
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < DPL; ++e) s = fmaf(x[e], y[e], s);
  s = sum16(s);
  if (sub == 0) stat[rh] = make_float2(lse[rh] * kLog2e, s);
}

// With the compact layout two workgroups fit a CU: registers for two
// wavefronts per SIMD (256 each); otherwise one.
template <int D, int CT>
__global__ __launch_bounds__(256, bwd_compact(CT * 32) ? 2 : 1) void attn_bwd_block_kernel(
    AttnBwdArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dO, const float2* __restrict__ stat, const int32_t* __restrict__ offs,
    const int32_t* __restrict__ toffs, int64_t ncl, const int32_t* __restrict__ pairs, uint16_t* __restrict__ part_dq,
    float* __restrict__ dk_acc, float* __restrict__ dv_acc, uint16_t* __restrict__ dk_out,
    uint16_t* __restrict__ dv_out) {
  constexpr int KS = D / 32;      // 32-dim k-steps of S^T and dP^T
  constexpr int LDK = D + 8;      // padded K / V row (bf16)
  constexpr int C = CT * 32;      // keys per block
  constexpr int MT = C / 16;      // 16-key tiles
  constexpr int DT = D / 16;      // 16-dim tiles
  constexpr int DTW = DT / 4;     // 16-dim tiles of dK, dV per wavefront
  constexpr int LPK = C + 8;         // padded P / dS row (bf16, one row per column, keys along it)
  constexpr int LQC = D + 8;         // padded q / do row (bf16, one row per column)
  constexpr bool CMP = bwd_compact(C);
  constexpr int NCD = D / 8, NCC = C / 8;  // 16-byte chunks per row of D / of C elements
  constexpr int RW = bwd_region(C, D);     // compact: elements of a wavefront's P + dS (+ dq staging) region
  extern __shared__ __align__(16) uint16_t lds[];
  // padded: K, V [C][LDK]; P, dS [64][LPK]; q, do [64][LQC]; dq staging [4][16][LQC]
  // compact: K, V [C][D]; q, do [64][D]; then per wavefront [P 16 x C][dS 16 x C],
  // whose first 16 x D elements also hold that wavefront's dq staging rows
  uint16_t* kl = lds;
  uint16_t* vl = kl + C * (CMP ? D : LDK);
  uint16_t* qr = vl + C * (CMP ? D : LDK);
  uint16_t* dr = qr + kBwdCols * (CMP ? D : LQC);
  uint16_t* pt = dr + kBwdCols * (CMP ? D : LQC);       // padded: P; compact: the wavefront regions
  uint16_t* st = pt + (CMP ? 0 : kBwdCols * LPK);       // padded: dS
  uint16_t* tb = CMP ? pt + (threadIdx.x >> 6) * RW : st + kBwdCols * LPK + (threadIdx.x >> 6) * 16 * LQC;
  // element e (a multiple of 4) of row r of each tile
  auto at_kv = [&](uint16_t* base, int r, int e) {
    return CMP ? base + r * D + (((e >> 3) ^ bwd_swz_rows<NCD>(r)) << 3) + (e & 7) : base + r * LDK + e;
  };
  auto at_qd = [&](uint16_t* base, int r, int e) {
    return CMP ? base + r * D + (((e >> 3) ^ bwd_swz_cols<NCD>(r)) << 3) + (e & 7) : base + r * LQC + e;
  };
  auto at_ps = [&](bool ds, int r, int e) {
    return CMP ? pt + (r >> 4) * RW + (ds ? 16 * C : 0) + (r & 15) * C + (((e >> 3) ^ bwd_swz_cols<NCC>(r)) << 3) +
                     (e & 7)
               : (ds ? st : pt) + r * LPK + e;
  };
  auto at_tb = [&](int r, int e) {
    return CMP ? tb + r * D + (((e >> 3) ^ bwd_swz_rows<NCD>(r)) << 3) + (e & 7) : tb + r * LQC + e;
  };

  int64_t cl;
  int beg, end;
  if (!cluster_chunk(offs, toffs, ncl, blockIdx.x, kBwdChunk, cl, beg, end)) return;
  const int bh = static_cast<int>(cl / a.M1);
  const int blk = static_cast<int>(cl - static_cast<int64_t>(bh) * a.M1);
  const int b = bh / a.Hkv, h = bh - b * a.Hkv;
  const int r0 = blk * C;
  const int nkeys = min(C, a.N - r0);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, grp = lane >> 4;

  const uint16_t* kb = k + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  const uint16_t* vb = v + (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  for (int e = threadIdx.x; e < C * (D / 8); e += 256) {
    const int r = e / (D / 8), c8 = (e - r * (D / 8)) * 8;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (r < nkeys) {
      kv = *reinterpret_cast<const uint4*>(kb + static_cast<int64_t>(r) * D + c8);
      vv = *reinterpret_cast<const uint4*>(vb + static_cast<int64_t>(r) * D + c8);
    }
    *reinterpret_cast<uint4*>(at_kv(kl, r, c8)) = kv;
    *reinterpret_cast<uint4*>(at_kv(vl, r, c8)) = vv;
  }

  // dV, dK of this wavefront's dims: [key tile][dim tile j: dt = wave*DTW + j]
  f32x4b2 accv[MT][DTW], acck[MT][DTW];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int jj = 0; jj < DTW; ++jj) {
      accv[mt][jj] = f32x4b2{0.f, 0.f, 0.f, 0.f};
      acck[mt][jj] = f32x4b2{0.f, 0.f, 0.f, 0.f};
    }

  const int ncols = (end - beg) * a.G;
  for (int g0 = 0; g0 < ncols; g0 += kBwdCols) {
    const int cidx = g0 + wave * 16 + col;  // this lane's (pair, head) column
    const bool valid = cidx < ncols;
    const int j = valid ? cidx / a.G : 0, hh = valid ? cidx - j * a.G : 0;
    const int pr = valid ? pairs[beg + j] : -1;
    const int rr = pr >= 0 ? pr >> 8 : 0, slot = pr & 255;
    const int row = a.row0 + rr;
    const int t = a.N - a.Nq + row;
    const int kmax = pr < 0 ? 0 : (a.causal ? min(nkeys, t - r0 + 1) : nkeys);
    const int64_t qrow = ((static_cast<int64_t>(b) * a.H + h * a.G + hh) * a.Nq + row);
    bf16x8b2 qb[KS], db[KS];
    {
      const uint16_t* qp = q + qrow * D + grp * 8;
      const uint16_t* dp = dO + qrow * D + grp * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 uq = make_uint4(0, 0, 0, 0), ud = make_uint4(0, 0, 0, 0);
        if (pr >= 0) {
          uq = *reinterpret_cast<const uint4*>(qp + ks * 32);
          ud = *reinterpret_cast<const uint4*>(dp + ks * 32);
        }
        qb[ks] = u4_bf16x8b2(uq);
        db[ks] = u4_bf16x8b2(ud);
        // the group's q and do rows for the dK / dV products
        *reinterpret_cast<uint4*>(at_qd(qr, wave * 16 + col, ks * 32 + grp * 8)) = uq;
        *reinterpret_cast<uint4*>(at_qd(dr, wave * 16 + col, ks * 32 + grp * 8)) = ud;
      }
    }
    const float2 sd = pr >= 0 ? stat[qrow] : make_float2(0.f, 0.f);
    // P^T and dS^T tiles: tile mt holds keys mt*16 + 4*grp + i of column `col`
    float pv[MT][4], dsv[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      f32x4b2 sacc = {0.f, 0.f, 0.f, 0.f}, pacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const uint4 ka = *reinterpret_cast<const uint4*>(at_kv(kl, mt * 16 + col, ks * 32 + grp * 8));
        const uint4 va = *reinterpret_cast<const uint4*>(at_kv(vl, mt * 16 + col, ks * 32 + grp * 8));
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(u4_bf16x8b2(ka), qb[ks], sacc, 0, 0, 0);
        pacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(u4_bf16x8b2(va), db[ks], pacc, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = mt * 16 + 4 * grp + i;
        const float p = key < kmax ? fast_exp2(sacc[i] * a.qscale2 - sd.x) : 0.f;
        pv[mt][i] = p;
        dsv[mt][i] = p * (pacc[i] - sd.y);
      }
    }
    // dq^T = K^T dS^T (the operand key order of the forward's O^T = V^T P)
    f32x4b2 qacc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) qacc[dt] = f32x4b2{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < MT / 2; ++s2) {
      uint4 u;
      u.x = pack2_bf16(dsv[2 * s2][0], dsv[2 * s2][1]);
      u.y = pack2_bf16(dsv[2 * s2][2], dsv[2 * s2][3]);
      u.z = pack2_bf16(dsv[2 * s2 + 1][0], dsv[2 * s2 + 1][1]);
      u.w = pack2_bf16(dsv[2 * s2 + 1][2], dsv[2 * s2 + 1][3]);
      const bf16x8b2 sb = u4_bf16x8b2(u);
      // K^T operand from the row-major K: keys 32 s2 + 4 grp + 0..3 and
      // 32 s2 + 16 + 4 grp + 0..3 (dS's operand order) of dim dt*16 + col,
      // by transposing reads (lane col: key row 4 grp + col / 4, dims 4 (col % 4))
      const int kr = 32 * s2 + 4 * grp + col / 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const v4s16 lo = lds_read_tr16x4(at_kv(kl, kr, dt * 16 + 4 * (col & 3)));
        const v4s16 hi = lds_read_tr16x4(at_kv(kl, kr + 16, dt * 16 + 4 * (col & 3)));
        const bf16x8b2 ak = __builtin_bit_cast(bf16x8b2, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        qacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, sb, qacc[dt], 0, 0, 0);
      }
    }
    {
      // the 16 dq partial rows of this wavefront through LDS, stored as whole
      // rows (16 lanes x 16 bytes per row)
      const int64_t pidx = ((static_cast<int64_t>(bh) * a.nrows + rr) * a.K + slot) * a.G + hh;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        uint2 w;
        w.x = pack2_bf16(qacc[dt][0] * a.rscale, qacc[dt][1] * a.rscale);
        w.y = pack2_bf16(qacc[dt][2] * a.rscale, qacc[dt][3] * a.rscale);
        *reinterpret_cast<uint2*>(at_tb(col, dt * 16 + 4 * grp)) = w;
      }
      wave_sync();
#pragma unroll
      for (int u = 0; u < 16 * D / 8 / 64; ++u) {
        const int e = u * 64 + lane;
        const int r = e / (D / 8), c8 = (e - r * (D / 8)) * 8;
        const int64_t px = __shfl(pidx, r);  // lanes 0-15 hold columns 0-15
        const bool ok = __shfl(pr, r) >= 0;
        const uint4 x = *reinterpret_cast<const uint4*>(at_tb(r, c8));
        if (ok) *reinterpret_cast<uint4*>(part_dq + px * D + c8) = x;
      }
      wave_sync();
    }
    // P and dS of the group, one row per column (this lane's 4 keys of each
    // 16-key tile in one 8-byte store)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      *reinterpret_cast<uint2*>(at_ps(false, wave * 16 + col, mt * 16 + 4 * grp)) =
          make_uint2(pack2_bf16(pv[mt][0], pv[mt][1]), pack2_bf16(pv[mt][2], pv[mt][3]));
      *reinterpret_cast<uint2*>(at_ps(true, wave * 16 + col, mt * 16 + 4 * grp)) =
          make_uint2(pack2_bf16(dsv[mt][0], dsv[mt][1]), pack2_bf16(dsv[mt][2], dsv[mt][3]));
    }
    __syncthreads();
    // dV[key][d] += sum_c P^T[key][c] do[c][d];  dK[key][d] += sum_c dS^T[key][c] q[c][d]
    // Every operand below holds 8 consecutive columns kk*32 + 8 grp + 0..7 of
    // one key (P, dS) or one dim (do, q): two transposing reads of 4 rows,
    // lane col reading row 8 grp + col / 4 (+4) at element 4 (col % 4).
#pragma unroll
    for (int kk = 0; kk < kBwdCols / 32; ++kk) {
      const int ar = kk * 32 + 8 * grp + col / 4;
      const int ae = 4 * (col & 3);
      auto join = [](v4s16 lo, v4s16 hi) {
        return __builtin_bit_cast(bf16x8b2, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      bf16x8b2 bdo[DTW], bq[DTW];
#pragma unroll
      for (int jj = 0; jj < DTW; ++jj) {
        const int e = (wave * DTW + jj) * 16 + ae;
        bdo[jj] = join(lds_read_tr16x4(at_qd(dr, ar, e)), lds_read_tr16x4(at_qd(dr, ar + 4, e)));
        bq[jj] = join(lds_read_tr16x4(at_qd(qr, ar, e)), lds_read_tr16x4(at_qd(qr, ar + 4, e)));
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int e = mt * 16 + ae;
        const bf16x8b2 ap = join(lds_read_tr16x4(at_ps(false, ar, e)), lds_read_tr16x4(at_ps(false, ar + 4, e)));
        const bf16x8b2 as = join(lds_read_tr16x4(at_ps(true, ar, e)), lds_read_tr16x4(at_ps(true, ar + 4, e)));
#pragma unroll
        for (int jj = 0; jj < DTW; ++jj) {
          accv[mt][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap, bdo[jj], accv[mt][jj], 0, 0, 0);
          acck[mt][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as, bq[jj], acck[mt][jj], 0, 0, 0);
        }
      }
    }
    __syncthreads();  // the group's LDS rows are read before the next group writes them
  }

  // accv[mt][jj][i]: key mt*16 + 4*grp + i, dim (wave*DTW + jj)*16 + col
  if (a.direct && toffs[cl + 1] - toffs[cl] == 1) {
    // the block's only chunk: dV, dK in the problem dtype, two dims per
    // 4-byte store (even lanes dV, odd lanes dK, each with its neighbour's value)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = mt * 16 + 4 * grp + i;
        if (key >= nkeys) continue;  // the same for both lanes of a pair
        const int64_t base = (static_cast<int64_t>(bh) * a.Nkv + r0 + key) * D;
#pragma unroll
        for (int jj = 0; jj < DTW; ++jj) {
          const int dcol = (wave * DTW + jj) * 16 + (col & ~1);
          const float vv = accv[mt][jj][i], kv = acck[mt][jj][i] * a.rscale;
          const float vn = __shfl_xor(vv, 1), kn = __shfl_xor(kv, 1);
          if (col & 1)
            *reinterpret_cast<uint32_t*>(dk_out + base + dcol) = pack2_bf16(kn, kv);
          else
            *reinterpret_cast<uint32_t*>(dv_out + base + dcol) = pack2_bf16(vv, vn);
        }
      }
    return;
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = mt * 16 + 4 * grp + i;
      if (key >= nkeys) continue;
      const int64_t base = (static_cast<int64_t>(bh) * a.Nkv + r0 + key) * D;
#pragma unroll
      for (int jj = 0; jj < DTW; ++jj) {
        const int dcol = (wave * DTW + jj) * 16 + col;
        atomicAdd(dv_acc + base + dcol, accv[mt][jj][i]);
        atomicAdd(dk_acc + base + dcol, acck[mt][jj][i] * a.rscale);
      }
    }
}

// dq of each (row of the chunk, query head): the sum of its slots' partials.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(AttnBwdArgs a, const int32_t* __restrict__ idx,
                                                          const uint16_t* __restrict__ part_dq,
                                                          uint16_t* __restrict__ dq) {
  constexpr int DPL = D / 16;
  const int sub = threadIdx.x & 15;
  const int rr = blockIdx.x * 16 + (threadIdx.x >> 4);
  if (rr >= a.nrows) return;
  const int hq = blockIdx.y % a.H;
  const int b = blockIdx.y / a.H;
  const int hk = hq / a.G, hh = hq - hk * a.G;
  const int bh = b * a.Hkv + hk;
  const int row = a.row0 + rr;
  const int32_t* sel = idx + (static_cast<int64_t>(bh) * a.Nq + row) * a.K;
  float acc[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
  // four slots' indices, then their partials, requested together (the sum
  // keeps the slot order)
  constexpr int SB = 4;
  const int64_t pbase = (static_cast<int64_t>(bh) * a.nrows + rr) * a.K;
  for (int s0 = 0; s0 < a.K; s0 += SB) {
    bool use[SB];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int x = s0 + u < a.K ? sel[s0 + u] : -1;
      use[u] = x >= 0 && x < a.M1;  // padding: no partial was written
    }
    float x[SB][DPL];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      if (use[u]) {
        load_row_part<uint16_t, DPL>(part_dq + ((pbase + s0 + u) * a.G + hh) * D + sub * DPL, x[u]);
      } else {
#pragma unroll
        for (int e = 0; e < DPL; ++e) x[u][e] = 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      if (!use[u]) continue;
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] += x[u][e];
    }
  }
  const int64_t orow = (static_cast<int64_t>(b) * a.H + hq) * a.Nq + row;
  store_bf16_part<DPL>(dq + orow * D + sub * DPL, acc);
}

// dk, dv [B, Hkv, N (row stride Nkv), D] from the fp32 accumulators.
__global__ __launch_bounds__(256) void attn_bwd_finalize_kernel(const float* __restrict__ dk_acc,
                                                                const float* __restrict__ dv_acc,
                                                                uint16_t* __restrict__ dk, uint16_t* __restrict__ dv,
                                                                int64_t n4) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n4) return;
  const float4 x = reinterpret_cast<const float4*>(dk_acc)[i];
  const float4 y = reinterpret_cast<const float4*>(dv_acc)[i];
  reinterpret_cast<uint2*>(dk)[i] = make_uint2(pack2_bf16(x.x, x.y), pack2_bf16(x.z, x.w));
  reinterpret_cast<uint2*>(dv)[i] = make_uint2(pack2_bf16(y.x, y.y), pack2_bf16(y.z, y.w));
}

__global__ __launch_bounds__(256) void fill_zero_f32_kernel(float* p, int64_t n) {
  for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < n; i += 256LL * gridDim.x) p[i] = 0.f;
}

// Direct launches: one wavefront per (batch x KV head, key block), from the
// cluster's chunk offsets.  Before the block kernel: the fp32 accumulator rows
// of blocks with several chunks are cleared.  After it: those rows go to the
// problem dtype, and blocks no pair selected get zero rows (a block with one
// chunk was written by the block kernel itself).
template <int D, bool AFTER>
__global__ __launch_bounds__(256) void attn_bwd_blocks_kernel(AttnBwdArgs a, int BH, const int32_t* __restrict__ toffs,
                                                              float* __restrict__ dk_acc, float* __restrict__ dv_acc,
                                                              uint16_t* __restrict__ dk, uint16_t* __restrict__ dv) {
  const int64_t w = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (w >= static_cast<int64_t>(BH) * a.M1) return;
  const int lane = threadIdx.x & 63;
  const int nch = toffs[w + 1] - toffs[w];
  if (nch == 1 || (!AFTER && nch == 0)) return;
  const int bh = static_cast<int>(w / a.M1), blk = static_cast<int>(w - static_cast<int64_t>(bh) * a.M1);
  const int r0 = blk * a.C;
  const int64_t e0 = (static_cast<int64_t>(bh) * a.Nkv + r0) * D;
  const int n4 = min(a.C, a.N - r0) * D / 4;  // float4 groups of the block's rows
  for (int e = lane; e < n4; e += 64) {
    if constexpr (!AFTER) {
      reinterpret_cast<float4*>(dk_acc + e0)[e] = make_float4(0.f, 0.f, 0.f, 0.f);
      reinterpret_cast<float4*>(dv_acc + e0)[e] = make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f), y = x;
      if (nch > 1) {
        x = reinterpret_cast<const float4*>(dk_acc + e0)[e];
        y = reinterpret_cast<const float4*>(dv_acc + e0)[e];
      }
      reinterpret_cast<uint2*>(dk + e0)[e] = make_uint2(pack2_bf16(x.x, x.y), pack2_bf16(x.z, x.w));
      reinterpret_cast<uint2*>(dv + e0)[e] = make_uint2(pack2_bf16(y.x, y.y), pack2_bf16(y.z, y.w));
    }
  }
}

// Zero rows [N, Nkv) of every (batch, KV head) of dk and dv.
template <int D>
__global__ __launch_bounds__(256) void attn_bwd_tail_kernel(int BH, int N, int Nkv, uint16_t* __restrict__ dk,
                                                            uint16_t* __restrict__ dv) {
  const int64_t per = static_cast<int64_t>(Nkv - N) * D / 4;  // uint2 groups per head
  for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < BH * per; i += 256LL * gridDim.x) {
    const int64_t bh = i / per, e = i - bh * per;
    const int64_t off = (bh * Nkv + N) * D / 4 + e;
    reinterpret_cast<uint2*>(dk)[off] = make_uint2(0u, 0u);
    reinterpret_cast<uint2*>(dv)[off] = make_uint2(0u, 0u);
  }
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------

bool attn_bwd_supported(const Shape& s) {
  return s.bf16 && (s.D == 64 || s.D == 128) && (s.C == 32 || s.C == 64 || s.C == 96 || s.C == 128) &&
         s.K <= 256;
}

constexpr size_t kBwdPartialBudget = size_t(4) << 30;

static int bwd_chunk_rows(const Shape& s) {
  const size_t per_row = static_cast<size_t>(s.BH()) * s.K * s.G * s.D * 2;
  return static_cast<int>(std::min<size_t>(s.Nq, std::max<size_t>(kBwdPartialBudget / per_row, 1)));
}

struct BwdWs {
  size_t stat, dk, dv, part, cl, total;
};

static BwdWs bwd_layout(const Shape& s, const Geo& geo) {
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  const size_t ch = bwd_chunk_rows(s);
  const size_t np = static_cast<size_t>(s.BH()) * ch * s.K;
  const size_t kv = static_cast<size_t>(s.BH()) * s.Nkv * s.D * 4;
  BwdWs w{};
  size_t o = 0;
  w.stat = o; o += al(static_cast<size_t>(s.B) * s.H * s.Nq * 8);
  w.dk = o;   o += al(kv);
  w.dv = o;   o += al(kv);
  w.part = o; o += al(np * s.G * s.D * 2);
  w.cl = o;   o += al(cluster_ws(s.BH(), geo.M[1], static_cast<int64_t>(np), static_cast<int>(ch)));
  w.total = o;
  return w;
}

size_t attn_bwd_ws(const Shape& s, const Geo& geo) { return bwd_layout(s, geo).total; }

template <int D>
static hipError_t launch_bwd_d(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                               const int32_t* idx, const void* o, const float* lse, const void* d_o, void* dq,
                               void* dk, void* dv, void* ws, hipStream_t st) {
  const BwdWs w = bwd_layout(s, geo);
  char* base = static_cast<char*>(ws);
  float2* stat = reinterpret_cast<float2*>(base + w.stat);
  float* dk_acc = reinterpret_cast<float*>(base + w.dk);
  float* dv_acc = reinterpret_cast<float*>(base + w.dv);
  uint16_t* part = reinterpret_cast<uint16_t*>(base + w.part);
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  const uint16_t* dd = static_cast<const uint16_t*>(d_o);
  AttnBwdArgs a{s.H, s.Hkv, s.G, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], 0, s.Nq,
                kLog2e / sqrtf(static_cast<float>(s.D)), 1.0f / sqrtf(static_cast<float>(s.D)), s.Nkv};
  hipError_t e;
  const int64_t nkv = static_cast<int64_t>(s.BH()) * s.Nkv * D;
  const int ch = bwd_chunk_rows(s);
  a.direct = ch >= s.Nq ? 1 : 0;
  const int64_t nblk = static_cast<int64_t>(s.BH()) * geo.M[1];
  uint16_t* dk16 = static_cast<uint16_t*>(dk);
  uint16_t* dv16 = static_cast<uint16_t*>(dv);
  {
    ProfScope ps("attn_bwd_prep", st);
    if (!a.direct) {
      fill_zero_f32_kernel<<<static_cast<unsigned>(std::min<int64_t>((nkv + 255) / 256, 8192)), 256, 0, st>>>(
          dk_acc, nkv);
      fill_zero_f32_kernel<<<static_cast<unsigned>(std::min<int64_t>((nkv + 255) / 256, 8192)), 256, 0, st>>>(
          dv_acc, nkv);
    }
    const int64_t nrh = static_cast<int64_t>(s.B) * s.H * s.Nq;
    attn_bwd_prep_kernel<D><<<static_cast<unsigned>((nrh + 15) / 16), 256, 0, st>>>(
        a, static_cast<const uint16_t*>(o), dd, lse, stat, nrh);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  ClusterOut co{};
  for (int row0 = 0; row0 < s.Nq; row0 += ch) {
    const int nrows = std::min(ch, s.Nq - row0);
    a.row0 = row0;
    a.nrows = nrows;
    ClusterArgs ca{idx, nullptr, s.K, s.Nq, s.N, s.C, s.K, s.causal, geo.M[1], kClusterAttn, row0, nrows, s.g};
    if ((e = launch_cluster(ca, s.BH(), base + w.cl, &co, st, kBwdChunk)) != hipSuccess) return e;
    if (a.direct) {
      ProfScope ps("attn_bwd_prep", st);
      attn_bwd_blocks_kernel<D, false><<<static_cast<unsigned>((nblk + 3) / 4), 256, 0, st>>>(
          a, s.BH(), co.toffs, dk_acc, dv_acc, dk16, dv16);
    }
    {
      ProfScope ps("attn_bwd_block", st);
      const int64_t np = static_cast<int64_t>(s.BH()) * nrows * s.K;
      dim3 grid(static_cast<unsigned>(cluster_max_chunks(s.BH(), geo.M[1], np, kBwdChunk)));
      const size_t lds = bwd_lds_elems(s.C, D) * 2;
      auto go = [&](auto kern) {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                  static_cast<int>(lds));
        kern<<<grid, 256, lds, st>>>(a, qq, kk, vv, dd, stat, co.offs, co.toffs, co.ncl, co.pairs, part, dk_acc,
                                     dv_acc, dk16, dv16);
      };
      if (s.C == 32)
        go(attn_bwd_block_kernel<D, 1>);
      else if (s.C == 64)
        go(attn_bwd_block_kernel<D, 2>);
      else if (s.C == 96)
        go(attn_bwd_block_kernel<D, 3>);
      else
        go(attn_bwd_block_kernel<D, 4>);
    }
    {
      ProfScope ps("attn_bwd_dq", st);
      dim3 grid(static_cast<unsigned>((nrows + 15) / 16), s.B * s.H);
      attn_bwd_dq_kernel<D><<<grid, 256, 0, st>>>(a, idx, part, static_cast<uint16_t*>(dq));
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  {
    ProfScope ps("attn_bwd_finalize", st);
    if (a.direct) {
      attn_bwd_blocks_kernel<D, true><<<static_cast<unsigned>((nblk + 3) / 4), 256, 0, st>>>(
          a, s.BH(), co.toffs, dk_acc, dv_acc, dk16, dv16);
      if (s.Nkv > s.N) {
        const int64_t tail = static_cast<int64_t>(s.BH()) * (s.Nkv - s.N) * D / 4;
        attn_bwd_tail_kernel<D><<<static_cast<unsigned>(std::min<int64_t>((tail + 255) / 256, 8192)), 256, 0, st>>>(
            s.BH(), s.N, s.Nkv, dk16, dv16);
      }
    } else {
      const int64_t n4 = nkv / 4;
      attn_bwd_finalize_kernel<<<static_cast<unsigned>((n4 + 255) / 256), 256, 0, st>>>(dk_acc, dv_acc, dk16, dv16,
                                                                                         n4);
    }
  }
  return hipGetLastError();
}

hipError_t launch_attention_bwd(const Shape& s, const Geo& geo, const void* q, const void* k, const void* v,
                                const int32_t* idx, const void* o, const float* lse, const void* d_o, void* dq,
                                void* dk, void* dv, void* ws, hipStream_t st) {
  return s.D == 128 ? launch_bwd_d<128>(s, geo, q, k, v, idx, o, lse, d_o, dq, dk, dv, ws, st)
                    : launch_bwd_d<64>(s, geo, q, k, v, idx, o, lse, d_o, dq, dk, dv, ws, st);
}

}  // namespace pisa
