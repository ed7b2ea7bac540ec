// Step 1: strided antidiagonal block scoring (XAttention Sec. 3.2, Algorithm 1).
//
// The reshapes of Algorithm 1 make reduced row R of Q~ the concatenation
// (along features) of query rows R*S + S-1, ..., R*S and reduced column c of
// K~ the concatenation of key rows c*S, ..., c*S + S-1, so
//   X[R][c] = q~_R . k~_c = sum_{t<S} q[R*S + S-1-t] . k[c*S + t],
// the sum over the antidiagonal of the S x S sub-block (R, c) of Q K^T.
// K~ is a plain view of K ([L/S][S*d], row c at K + c*S*d) and Q~ a view of Q
// with the S sub-rows reversed: no data is moved to build either.
//
// Kernel score_partials computes X^T = K~ Q~^T in 256 x 256 tiles on bf16
// MFMA (fp32 accumulate; 8 waves of 128 columns x 64 rows; 64-deep K chunks
// streamed by direct-to-LDS loads through a two-stage pipeline) and, in its
// epilogue, per reduced row R and 128-column sub-tile t: the sub-tile max m
// (log2 domain), l = sum exp2(x - m), and per key block j the partial mass
// sum_{c in j} exp2(x - m). Kernel score_finalize
// merges the tiles of each row (m_R = max_t m, l_R = sum_t l 2^(m - m_R)),
// normalises, and averages the B/S reduced rows of each query block.
#include <atomic>

#include "common.h"
#include "score_rows.h"

using namespace xattn;

namespace {

constexpr int TM = 256;             // reduced rows (R) and columns (c) per workgroup tile
constexpr int TSUB = kTsub;         // column sub-tile owning one (m, l) pair per row
constexpr int KC = 64;              // reduced-K chunk per pipeline stage (128-byte rows)
constexpr int NSTAGE = 2;           // stages: one chunk computed while the next loads
constexpr int kThreads = 512;       // 8 waves: 2 (columns) x 4 (rows), 128 c x 64 R each
constexpr int kStage = TM * KC;     // bf16 elements of one operand in one stage
constexpr int kCPR = KC / 8;        // 16-byte chunks per LDS row
constexpr int kRowsPer256 = 128 / KC;  // LDS rows per 256-byte bank period
constexpr int kDmaRows = 512 / KC;  // rows one 1 KB direct-to-LDS instruction fills
constexpr int kDmaPerOp = 32 / kDmaRows;  // instructions per wave per operand per chunk
static_assert(NSTAGE * 2 * kStage * 2 <= 160 * 1024, "LDS budget");

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

__device__ __forceinline__ void tri_decode(int t, int& rt, int& ct) {
  int r = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while (r * (r + 1) / 2 > t) --r;
  while ((r + 1) * (r + 2) / 2 <= t) ++r;
  rt = r;
  ct = t - r * (r + 1) / 2;
}

// LDS rows hold KC bf16 (kCPR chunks of 16 B); chunk c of row r sits at
// position c ^ ((r / kRowsPer256) mod kCPR), so 16 consecutive rows read at
// one logical chunk hit 16 distinct bank groups.
__device__ __forceinline__ int swz_row(int r) { return (r / kRowsPer256) & (kCPR - 1); }

// Lane l < 32 returns a[l] + a[l + 32]; lane l >= 32 returns b[l - 32] + b[l]
// (one v_permlane32_swap exchanges the upper half of a with the lower half of
// b).
__device__ __forceinline__ float half_pair_sum(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, a),
                                                  __builtin_bit_cast(uint32_t, b), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

// NRB = reduced rows (and columns) per 128-token block = 128 / S.
template <int NRB, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 1) void score_partials(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int hq, int hkv, int L,
    int NR, int NB, int NT, int tiles_per_head, int n_work, float scale_log2,
    SubRowPairing pairing, float* __restrict__ part, float2* __restrict__ stats) {
  constexpr int S = kBlock / NRB;
  constexpr int KD = S * kHeadDim;  // reduced inner dimension S*d
  constexpr int NCH = KD / KC;      // >= 2 (S >= 1)
  // [stage][operand A = K~ rows (c) | B = Q~ rows (R)][256 rows x 32]
  __shared__ __attribute__((aligned(1024))) uint16_t lds[NSTAGE * 2 * kStage];

  const int tid = threadIdx.x, lane = tid & 63, lr = lane & 31, lh = lane >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wc = wv & 1, wr = wv >> 1;

  // Persistent: each workgroup runs a sequence of tiles. Logical order
  // (kv head, row tile, column tile, query head in group); XCD x (blockIdx %
  // 8) takes one contiguous range of it, so the heads of a group that share
  // K~ rows run on one L2. While the last chunk of a tile is computed, the
  // first chunk of the next tile loads; its epilogue then overlaps that load.
  const int x8 = blockIdx.x % kNumXcd, k8 = blockIdx.x / kNumXcd;
  const int nper = gridDim.x / kNumXcd;  // workgroups per XCD (grid is a multiple of 8)
  const int per = n_work / kNumXcd, rem = n_work % kNumXcd;
  const int lo = x8 * per + (x8 < rem ? x8 : rem);
  const int cnt_x = per + (x8 < rem ? 1 : 0);
  const int G = hq / hkv;

  // The tile being loaded: its head, first reduced row / column, operand
  // bases (scalar) and this lane's load offsets. After a tile's last chunk
  // load it is switched to the next tile, whose first chunk then loads while
  // the finished tile (h_done, R0_done, c0_done) runs its epilogue.
  int th = 0, tR0 = 0, tc0 = 0;
  const uint16_t* tQh = q;
  const uint16_t* tKg = k;
  uint32_t offA[kDmaPerOp], offB[kDmaPerOp];
  auto load_tile = [&](int w) {
    const int hh = w % G;
    const int rest = w / G;
    const int tile = rest % tiles_per_head;
    const int gidx = rest / tiles_per_head;
    th = __builtin_amdgcn_readfirstlane((gidx / hkv) * hq + (gidx % hkv) * G + hh);
    int rt, ct;
    if (CAUSAL) {
      tri_decode(tile, rt, ct);
    } else {
      rt = tile / ceil_div(NR, TM);
      ct = tile % ceil_div(NR, TM);
    }
    tR0 = __builtin_amdgcn_readfirstlane(rt * TM);
    tc0 = __builtin_amdgcn_readfirstlane(ct * TM);
    tQh = q + (size_t)th * L * kHeadDim;
    tKg = k + (size_t)__builtin_amdgcn_readfirstlane(gidx) * L * kHeadDim;
    // direct-to-LDS staging: per stage each wave loads rows 32 wv .. +32 of
    // both operands, kDmaPerOp instructions (kDmaRows rows x 2 KC bytes)
    // each; rows beyond NR are clamped to NR - 1 (results masked / not stored)
#pragma unroll
    for (int i = 0; i < kDmaPerOp; ++i) {
      const int r = 32 * wv + kDmaRows * i + lane / kCPR;
      const int c = (lane & (kCPR - 1)) ^ swz_row(r);
      const int ra = min(tc0 + r, NR - 1), rb = min(tR0 + r, NR - 1);
      offA[i] = (uint32_t)(((size_t)ra * KD + c * 8) * 2);
      offB[i] = (uint32_t)(((size_t)rb * S * kHeadDim + c * 8) * 2);
    }
  };

  const uint32_t lds0 = XATTN_LDS_ADDR(lds);
  // lane t holds the query sub-row paired with key sub-row t; read per chunk
  // with v_readlane (a table lookup in kernel-argument memory would put a
  // scalar load and its wait on every chunk's critical path)
  const int qsub_lane = pairing.q[lane < S ? lane : 0];
  // Load pair i (operand A = K~ rows, B = Q~ rows) of chunk ch of tile t into
  // stage ch % NSTAGE.
  auto dma_pair = [&](int ch, int i) {
    const int kap0 = ch * KC;
    const uint16_t* baseA = tKg + kap0;
    const uint16_t* baseB =
        tQh + __builtin_amdgcn_readlane(qsub_lane, kap0 / kHeadDim) * kHeadDim + kap0 % kHeadDim;
    const uint32_t st = lds0 + (uint32_t)((ch % NSTAGE) * 2 * kStage * 2);
    const uint32_t row_lds = (uint32_t)((32 * wv + kDmaRows * i) * KC * 2);
    dma16(baseA, offA[i], st + row_lds);
    dma16(baseB, offB[i], st + kStage * 2 + row_lds);
  };

  f32x16 acc[4][2];

  // Diagonal tiles are computed in full (their masked half is ~2% of the MFMA
  // work of a causal layer); a per-MFMA skip would break the inner loop into
  // branches that serialise every LDS read with its MFMA.
  const uint32_t xa = (uint32_t)swz_row(lr);  // swizzle of this lane's rows (32 t, 64 wr: same)
  // hook(ks) runs at the start of k-step ks: the loads of the next chunk are
  // spread over the k-steps (a burst after the barrier stalls the wave at issue)
  auto compute = [&](int ch, auto hook) {
    const uint16_t* A = lds + (ch % NSTAGE) * 2 * kStage;
    const uint16_t* Bm = A + kStage;
#pragma unroll
    for (int ks = 0; ks < KC / 16; ++ks) {
      hook(ks);
      const uint32_t coff = (uint32_t)((((2 * ks + lh) ^ xa)) << 3);  // elements
      u32x4 bq[2];
#pragma unroll
      for (int n = 0; n < 2; ++n)
        bq[n] = *(const u32x4*)(Bm + (64 * wr + 32 * n + lr) * KC + coff);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const u32x4 ak = *(const u32x4*)(A + (128 * wc + 32 * t + lr) * KC + coff);
#pragma unroll
        for (int n = 0; n < 2; ++n) acc[t][n] = mfma32(as_bf16x8(ak), as_bf16x8(bq[n]), acc[t][n]);
      }
    }
    // Issue order per chunk: the 6 reads of k-step 0, then for each k-step its
    // 8 MFMAs with the 6 reads of the next k-step interleaved.
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int kk = 0; kk + 1 < KC / 16; ++kk) {
#pragma unroll
      for (int i = 0; i < 6; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
  };
  static_assert(kDmaPerOp == KC / 16, "one load pair per k-step");

  auto epilogue = [&](const int h, const int R0, const int c0) {
    // ---- epilogue per 32-row slab n: this lane owns reduced row R and 64 of the
    // wave's 128 columns; lane (lr, 1-lh) owns the other 64.
    const int csub = c0 + 128 * wc;  // first column of this wave's sub-tile
    const int tsub_idx = csub / TSUB;
    const int j0 = csub / NRB;
  #pragma unroll
    for (int n = 0; n < 2; ++n) {
      const int R = R0 + 64 * wr + 32 * n + lr;
      // Invalid columns (c > R when causal, c >= NR) occur only in sub-tiles
      // that reach past the slab's first row or the reduced length; the empty
      // asm keeps this uniform branch from becoming selects on every tile.
      const int Rslab = R0 + 64 * wr + 32 * n;
      if ((CAUSAL && csub + 127 > Rslab) || csub + 127 >= NR) {
        asm volatile("");
  #pragma unroll
        for (int t = 0; t < 4; ++t) {
  #pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int c = csub + 32 * t + 8 * (r >> 2) + 4 * lh + (r & 3);
            if (c >= NR || (CAUSAL && c > R)) acc[t][n][r] = -INFINITY;
          }
        }
      }
      // max of the raw products (the scale is positive), then every term as
      // one fma inside the exponential: p = 2^(x scale - m)
      float mloc = -INFINITY;
  #pragma unroll
      for (int t = 0; t < 4; ++t) {
  #pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, acc[t][n][r]);
      }
      const float m = fmaxf(mloc, __shfl_xor(mloc, 32)) * scale_log2;
      const float mref = (m == -INFINITY) ? 0.f : m;
      float gsum[16];  // groups of 4 consecutive columns: group gi = 4 t + r / 4
      float lloc = 0.f;
  #pragma unroll
      for (int t = 0; t < 4; ++t) {
  #pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          float sum = 0.f;
  #pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p = fast_exp2(fmaf(acc[t][n][4 * g4 + e], scale_log2, -mref));
            acc[t][n][4 * g4 + e] = p;
            sum += p;
          }
          gsum[4 * t + g4] = sum;
          lloc += sum;
        }
      }
      const float l = lloc + __shfl_xor(lloc, 32);
      const bool rvalid = R < NR;
      // part is [head][query block][key block][row in block] (causal: key
      // blocks <= the query block only, rows packed as a triangle): what the
      // finalize workgroup of one query block reads is one contiguous slab;
      // a half-wave writes 32 / NRB runs of NRB consecutive floats per block.
      const int Rv = rvalid ? R : 0;
      const int qb = Rv / NRB;
      float* pcol = part + part_row(h, qb, NB, CAUSAL) * NRB + (Rv % NRB);
      // key block j of this row is stored if it exists and, when causal, is
      // not above the diagonal (those are fully masked and have no slot)
      auto keep = [&](int j) { return rvalid && j < NB && (!CAUSAL || j <= qb); };
  
      if constexpr (NRB >= 8) {
        // group gi covers columns 8 gi + 4 lh + [0, 4): local block gi / (NRB / 8)
        constexpr int GPB = NRB / 8;
        constexpr int NBL = TSUB / NRB;
        auto block_sum = [&](int jb) {
          float sum = 0.f;
  #pragma unroll
          for (int x = 0; x < GPB; ++x) sum += gsum[jb * GPB + x];
          return sum;
        };
        if constexpr (NBL >= 2) {
          // blocks x and NBL/2 + x in one exchange: lanes < 32 end up with
          // block x's total over both column halves, lanes >= 32 with block
          // NBL/2 + x's, each the one it stores
  #pragma unroll
          for (int x = 0; x < NBL / 2; ++x) {
            const float tot = half_pair_sum(block_sum(x), block_sum(NBL / 2 + x));
            const int jb = lh * (NBL / 2) + x;
            if (keep(j0 + jb)) pcol[(size_t)(j0 + jb) * NRB] = tot;
          }
        } else {
          const float s0 = block_sum(0);
          const float tot = half_pair_sum(s0, s0);
          if (lh == 0 && keep(j0)) pcol[(size_t)j0 * NRB] = tot;
        }
      } else if constexpr (NRB == 4) {
        // each group of 4 columns is one block: local block 2 gi + lh
  #pragma unroll
        for (int gi = 0; gi < 16; ++gi) {
          const int j = j0 + 2 * gi + lh;
          if (keep(j)) pcol[(size_t)j * NRB] = gsum[gi];
        }
      } else {  // NRB == 2: each group holds two blocks
        static_assert(NRB == 2, "stride must divide the block");
  #pragma unroll
        for (int t = 0; t < 4; ++t) {
  #pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int gi = 4 * t + g4;
            const int j = j0 + 4 * gi + 2 * lh;
            if (keep(j)) pcol[(size_t)j * NRB] = acc[t][n][4 * g4] + acc[t][n][4 * g4 + 1];
            if (keep(j + 1))
              pcol[(size_t)(j + 1) * NRB] = acc[t][n][4 * g4 + 2] + acc[t][n][4 * g4 + 3];
          }
        }
      }
      // causal: a sub-tile starting after the row has no stats slot (all its
      // columns are masked for that row)
      if (rvalid && lh == 0 && tsub_idx < NT && (!CAUSAL || R >= tsub_idx * TSUB))
        stats[stats_at(h, tsub_idx, R, NR, NT, CAUSAL)] = make_float2(m, l);
    }
  };

  if (cnt_x <= k8) return;  // no tile for this workgroup (uniform)
  load_tile(lo + k8);
#pragma unroll
  for (int i = 0; i < kDmaPerOp; ++i) dma_pair(0, i);
  for (int it = k8; it < cnt_x; it += nper) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int n = 0; n < 2; ++n) acc[t][n] = f32x16{};
    // Step ch: this wave's loads of chunk ch have landed; the barrier makes
    // everyone's visible and ends every wave's reads of chunk ch - 1, whose
    // stage now receives chunk ch + 1, one pair per k-step of compute(ch).
    for (int ch = 0; ch + 1 < NCH; ++ch) {
      wait_vmcnt<0>();
      barrier_nofence();
      compute(ch, [&](int ks) { dma_pair(ch + 1, ks); });
    }
    wait_vmcnt<0>();
    barrier_nofence();
    // Chunk 0 of the next tile goes to stage 0 (chunk NCH - 2's, finished by
    // everyone) during the last chunk; after the last tile the same tile's
    // chunk 0 is loaded again (in bounds, never read).
    const int h_done = th, R0_done = tR0, c0_done = tc0;
    if (it + nper < cnt_x) load_tile(lo + it + nper);
    compute(NCH - 1, [&](int ks) { dma_pair(0, ks); });
    epilogue(h_done, R0_done, c0_done);
  }
  wait_vmcnt<0>();  // the last loads land before the LDS is released
}

// One workgroup (4 waves) per (query head, query block) row: the row's
// scores from its partial sums and tile statistics (finalize_row).
template <bool CAUSAL>
__global__ __launch_bounds__(kFinThreads) void score_finalize(const float* __restrict__ part,
                                                              const float2* __restrict__ stats,
                                                              int NR, int NB, int NT, int nrb,
                                                              float* __restrict__ scores) {
  __shared__ FinalizeLds lds;
  const int h = blockIdx.x / NB, b = blockIdx.x % NB;
  finalize_row<CAUSAL>(part, stats, NR, NB, NT, nrb, h, b, scores + ((size_t)h * NB + b) * NB,
                       lds);
}

// Compute units of the current device, rounded down to a multiple of the 8
// XCDs (cached per device).
int persistent_workgroups() {
  static std::atomic<int> cached[64];  // static storage: starts at zero
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  const bool cacheable = dev >= 0 && dev < 64;
  int n = cacheable ? cached[dev].load(std::memory_order_relaxed) : 0;
  if (n == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < kNumXcd)
      cus = 256;  // any multiple of 8 is a valid grid; this only sizes it
    n = cus / kNumXcd * kNumXcd;
    if (cacheable) cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <int NRB, bool CAUSAL>
hipError_t launch_partials(const void* q, const void* k, const XattnShape& s,
                           const SubRowPairing& pr, float* part, float* stats, hipStream_t st) {
  const int S = kBlock / NRB, NR = s.seq / S, NB = s.NB(), NT = ceil_div(NR, TSUB);
  const int T = ceil_div(NR, TM);
  const int tiles = CAUSAL ? T * (T + 1) / 2 : T * T;
  const int n_work = s.batch * s.hkv * tiles * (s.hq / s.hkv);
  const float scale_log2 = kLog2e / (sqrtf((float)kHeadDim) * (float)S);
  // one resident workgroup per CU (128 KB of LDS each), a multiple of 8
  const int wgs = persistent_workgroups();
  hipLaunchKernelGGL((score_partials<NRB, CAUSAL>), dim3(wgs), dim3(kThreads), 0, st,
                     (const uint16_t*)q, (const uint16_t*)k, s.hq, s.hkv, s.seq, NR, NB, NT,
                     tiles, n_work, scale_log2, pr, part, (float2*)stats);
  return hipGetLastError();
}

template <int NRB>
hipError_t launch_partials_c(const void* q, const void* k, const XattnShape& s,
                             const SubRowPairing& pr, float* part, float* stats, hipStream_t st) {
  return s.causal ? launch_partials<NRB, true>(q, k, s, pr, part, stats, st)
                  : launch_partials<NRB, false>(q, k, s, pr, part, stats, st);
}

}  // namespace

size_t score_scratch_bytes(const XattnShape& s, int stride) {
  const int NR = s.seq / stride, NB = s.NB(), NT = ceil_div(NR, TSUB);
  const size_t part = part_elems(s.HQ(), NB, kBlock / stride, s.causal) * sizeof(float);
  const size_t stats = (size_t)s.HQ() * stats_per_head(NR, NT, s.causal) * sizeof(float2);
  return ((part + 255) / 256) * 256 + stats;
}

ScoreScratch score_scratch_views(const XattnShape& s, int stride, void* scratch) {
  const size_t part_bytes =
      part_elems(s.HQ(), s.NB(), kBlock / stride, s.causal) * sizeof(float);
  ScoreScratch v;
  v.part = (float*)scratch;
  v.stats = (float*)((char*)scratch + ((part_bytes + 255) / 256) * 256);
  return v;
}

// The partial-sum kernel of xattn_score (the first of its two launches).
static hipError_t launch_score_partials(const void* q, const void* k, const XattnShape& s, int stride,
                                 const int32_t* qsub, void* scratch, hipStream_t st) {
  SubRowPairing pr;
  for (int t = 0; t < stride; ++t) pr.q[t] = qsub ? qsub[t] : stride - 1 - t;
  const ScoreScratch v = score_scratch_views(s, stride, scratch);
  switch (stride) {
    case 1: return launch_partials_c<128>(q, k, s, pr, v.part, v.stats, st);
    case 2: return launch_partials_c<64>(q, k, s, pr, v.part, v.stats, st);
    case 4: return launch_partials_c<32>(q, k, s, pr, v.part, v.stats, st);
    case 8: return launch_partials_c<16>(q, k, s, pr, v.part, v.stats, st);
    case 16: return launch_partials_c<8>(q, k, s, pr, v.part, v.stats, st);
    case 32: return launch_partials_c<4>(q, k, s, pr, v.part, v.stats, st);
    case 64: return launch_partials_c<2>(q, k, s, pr, v.part, v.stats, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_score(const void* q, const void* k, const XattnShape& s, int stride,
                        const int32_t* qsub, float* scores, void* scratch, hipStream_t st) {
  hipError_t e = launch_score_partials(q, k, s, stride, qsub, scratch, st);
  if (e != hipSuccess) return e;
  const int NR = s.seq / stride, NB = s.NB(), NT = ceil_div(NR, TSUB);
  const int nrb = kBlock / stride;
  const ScoreScratch v = score_scratch_views(s, stride, scratch);
  if (s.causal)
    hipLaunchKernelGGL(score_finalize<true>, dim3(s.HQ() * NB), dim3(kFinThreads), 0, st, v.part,
                       (const float2*)v.stats, NR, NB, NT, nrb, scores);
  else
    hipLaunchKernelGGL(score_finalize<false>, dim3(s.HQ() * NB), dim3(kFinThreads), 0, st,
                       v.part, (const float2*)v.stats, NR, NB, NT, nrb, scores);
  return hipGetLastError();
}
