// Plans, workspace layout and the device entry points of the C-ABI.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "internal.h"

namespace {

thread_local std::string g_detail;

int hip_status(int e) {
  if (e == hipSuccess) return FMM_OK;
  g_detail = hipGetErrorString(static_cast<hipError_t>(e));
  return FMM_ERR_HIP;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool is_gfx950(int dev) {
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return false;
  return std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
}

}  // namespace

struct fmm_plan {
  fmm::Problem pb;
  fmm::Workspace wl;
  fmm::DeviceTables tab;
  void *dev_tables;   // one device allocation backing tab
  int device;
};

extern "C" {

const char *fmm_status_string(int status) {
  switch (status) {
    case FMM_OK: return "ok";
    case FMM_ERR_ARG: return "invalid argument";
    case FMM_ERR_SHAPE: return "shape not divisible as required";
    case FMM_ERR_UNSUPPORTED: return "unsupported configuration";
    case FMM_ERR_NOT_EXACT: return "realization is not exact (Brent residual above tolerance)";
    case FMM_ERR_SINGULAR: return "singular basis change";
    case FMM_ERR_HIP: return "HIP runtime error";
    case FMM_ERR_DEVICE: return "device is not gfx950";
    case FMM_ERR_WORKSPACE: return "workspace too small or misaligned";
    case FMM_ERR_NOMEM: return "host allocation failed";
    default: return "unknown status";
  }
}

const char *fmm_last_error_detail(void) { return g_detail.c_str(); }

int fmm_device_check(int device) {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return FMM_ERR_HIP;
  return is_gfx950(device) ? FMM_OK : FMM_ERR_DEVICE;
}

int fmm_plan_create(const fmm_real *d, const fmm_plan_desc *desc, fmm_plan **out) {
  if (!out) return FMM_ERR_ARG;
  *out = nullptr;
  if (!d || !desc) return FMM_ERR_ARG;
  const fmm_plan_desc &q = *desc;
  constexpr int kFlags = FMM_FLAG_EXACT_DOT | FMM_FLAG_B_BLOCK128 | FMM_FLAG_B_BF16 | FMM_FLAG_LARGE_TILE;
  if ((q.flags & ~kFlags) != 0 || q.batch < 0 || q.M < 0 || q.K < 0 || q.N < 0) return FMM_ERR_ARG;
  if (q.depth < 1 || q.depth > fmm::kMaxDepth) return FMM_ERR_ARG;
  if (q.block != 16 && q.block != 32 && q.block != 128) return FMM_ERR_ARG;
  if (q.rule < FMM_RULE_FP32_AMAX || q.rule > FMM_RULE_POW2_OCP) return FMM_ERR_ARG;
  int sm = 2, sk = 2, sn = 2, sR = 0;
  if (fmm_realization_shape(d, &sm, &sk, &sn, &sR) != FMM_OK) return FMM_ERR_ARG;
  const bool shaped = !(sm == 2 && sk == 2 && sn == 2);
  if (shaped && (q.depth != 1 || (q.flags & (FMM_FLAG_B_BLOCK128 | FMM_FLAG_B_BF16))))
    return FMM_ERR_UNSUPPORTED;
  // the sub-block grid: 2^l x 2^l at <2,2,2>, m x k by k x n for other shapes
  const int64_t n = int64_t(1) << q.depth;
  const int64_t gm = shaped ? sm : n, gk = shaped ? sk : n, gn = shaped ? sn : n;
  if (q.M % gm || q.K % gk || q.N % gn) return FMM_ERR_SHAPE;
  if ((q.K / gk) % q.block) return FMM_ERR_SHAPE;
  // grid limits of the launches (batch on grid z/y, terms on grid y)
  if (q.batch > 65535) return FMM_ERR_UNSUPPORTED;
  // the weight-side deployment granularity is built for one level
  if ((q.flags & (FMM_FLAG_B_BLOCK128 | FMM_FLAG_B_BF16)) && q.depth != 1) return FMM_ERR_UNSUPPORTED;

  // the realization, as the C-ABI sees it
  int64_t R = 0, T = 0;
  const int rst = fmm_realization_terms(d, q.depth, &R, &T);
  if (rst != FMM_OK) return rst;

  // large-tile path: one or two levels, 256-row tiles, whole 64-byte (blocks
  // 16, 32) or 128-byte (block 128) K steps; E8M0 scales at blocks 32 and 128
  // on the fp8 matrix cores or (exact-dot flag) the folded-scale bf16 kernel,
  // fp32 scales and block 16 on the promote kernel.  It writes every P_r (4
  // bytes per output of each term) and reads it back, 8 / k' bytes per flop
  // against the fused path's none: plans with a fused kernel take it by
  // default where that round trip costs less than the fused path's smaller
  // tiles, k' >= 1024 (measured on both forms: the large tiles win at 1024
  // and above, lose at 512 and below); fp32 scales whenever the shape allows
  // (their fused promote kernel is slower at every measured k').
  // Plans of other shapes take it always (their W-combine fans each P_r out
  // to up to m n blocks of C), K = 0 included (C is then zero).
  const int64_t mp = q.M / gm, kp = q.K / gk, np = q.N / gn;
  const bool tiles_fit = mp % fmm::kSplitTile == 0 && np % fmm::kSplitTile == 0 &&
                         kp % (q.block == 128 ? 128 : 64) == 0 && kp < (int64_t(1) << 26) &&
                         q.batch * T * (mp / fmm::kSplitTile) * (np / fmm::kSplitTileN) < (int64_t(1) << 31);
  if (shaped && !tiles_fit) return FMM_ERR_UNSUPPORTED;
  const bool split_shape = q.depth <= 2 && kp > 0 && tiles_fit;

  fmm_plan *p = new (std::nothrow) fmm_plan;
  if (!p) return FMM_ERR_NOMEM;
  fmm::Problem &pb = p->pb;
  pb.batch = q.batch; pb.M = q.M; pb.K = q.K; pb.N = q.N;
  pb.depth = q.depth; pb.nsplit = (int)n;
  pb.mp = mp; pb.kp = kp; pb.np = np;
  pb.gm = (int)gm; pb.gk = (int)gk; pb.gn = (int)gn;
  pb.shaped = shaped ? 1 : 0;
  pb.block = q.block; pb.rule = q.rule;
  pb.R = (int)R; pb.T = T; pb.To = fmm::ipow(R, q.depth - 1);
  pb.kblocks = pb.kp / q.block;
  pb.scale_bytes = q.rule == FMM_RULE_FP32_AMAX ? 4 : 1;
  pb.exact_dot = (q.flags & FMM_FLAG_EXACT_DOT) ? 1 : 0;
  pb.b_rows = (q.flags & FMM_FLAG_B_BLOCK128) ? 128 : 1;
  pb.b_bf16 = (q.flags & FMM_FLAG_B_BF16) ? 1 : 0;
  // E8M0 scales have a fused 128 x 128 kernel: at blocks 32 and 128 on either
  // path (the fp8 matrix cores, or the exact-dot flag's folded-scale form),
  // at block 16 the folded-scale form (block 16 always runs exact-dot); fp32
  // scales only the large-tile exact-dot kernels
  const bool fused_exists = pb.scale_bytes == 1 && (q.block == 16 || q.block == 32 || q.block == 128);
  pb.split = shaped || (split_shape &&
             (!fused_exists || pb.kp >= fmm::kSplitMinK || (q.flags & FMM_FLAG_LARGE_TILE)));
  // fused 128 x 128 path: E8M0 scales at blocks 32 and 128 (the fp8 matrix
  // cores, or the exact-dot flag's folded-scale bf16 form) and block 16 (the
  // folded-scale form), whole 128-row tiles and 128-byte K steps
  const bool tile128 = fused_exists && pb.mp % 128 == 0 && pb.np % 128 == 0 && pb.kp > 0 &&
                       pb.kp % 128 == 0 && pb.kp < (int64_t(1) << 26);
  pb.layout = pb.split ? FMM_LAYOUT_TILE256x64 : tile128 ? FMM_LAYOUT_TILE128x128 : FMM_LAYOUT_ROWS;

  // workspace layout
  fmm::Workspace &wl = p->wl;
  size_t off = 0;
  const size_t B = (size_t)q.batch;
  wl.a_codes = off; off = align256(off + B * T * pb.mp * pb.kp);
  wl.b_codes = off; off = align256(off + B * T * pb.np * pb.kp);
  wl.a_scales = off; off = align256(off + B * T * fmm::scale_plane_bytes(pb, pb.mp));
  wl.b_scales = off; off = align256(off + B * T * fmm::scale_plane_bytes(pb, pb.np));
  wl.partial = off;
  if (q.depth >= 2 && !pb.split) off = align256(off + B * pb.To * 4 * pb.mp * pb.np * sizeof(float));
  wl.products = off;
  if (pb.split) off = align256(off + B * T * pb.mp * pb.np * sizeof(float));
  wl.b_amax = off;
  if (pb.b_rows > 1) off = align256(off + B * T * ((pb.np + 127) / 128) * pb.kblocks * sizeof(uint32_t));
  wl.total = off;

  // host tables: fp32 flattened U, V (dense rows; and their nonzeros in
  // ascending block order), base w, outer w.  Other shapes: the dense rows
  // and w padded with zeros to the kernels' grid capacities.
  const int nba = (int)(gm * gk), nbb = (int)(gk * gn), nbc = (int)(gm * gn);
  const int sta = shaped ? fmm::grid_capacity(nba) : nba, stb = shaped ? fmm::grid_capacity(nbb) : nbb;
  std::vector<float> U((size_t)T * sta, 0.0f), V((size_t)T * stb, 0.0f);
  std::vector<float> wfull;
  if (shaped) {
    std::vector<float> u0((size_t)T * nba), v0((size_t)T * nbb), w0((size_t)T * nbc);
    fmm_realization_tables(d, 1, u0.data(), v0.data(), w0.data());
    const int stc = fmm::grid_capacity(nbc);
    wfull.assign((size_t)T * stc, 0.0f);
    for (int64_t r = 0; r < T; ++r) {
      for (int b = 0; b < nba; ++b) U[r * sta + b] = u0[r * nba + b];
      for (int b = 0; b < nbb; ++b) V[r * stb + b] = v0[r * nbb + b];
      for (int b = 0; b < nbc; ++b) wfull[r * stc + b] = w0[r * nbc + b];
    }
  } else {
    fmm_realization_tables(d, q.depth, U.data(), V.data(), nullptr);
  }
  std::vector<int32_t> aoff(T + 1), boff(T + 1);
  std::vector<fmm::CoefEntry> aent, bent;
  for (int64_t r = 0; r < T; ++r) {
    aoff[r] = (int32_t)aent.size();
    boff[r] = (int32_t)bent.size();
    for (int b = 0; b < nba; ++b)
      if (U[r * sta + b] != 0.0f) aent.push_back({b, U[r * sta + b]});
    for (int b = 0; b < nbb; ++b)
      if (V[r * stb + b] != 0.0f) bent.push_back({b, V[r * stb + b]});
  }
  aoff[T] = (int32_t)aent.size();
  boff[T] = (int32_t)bent.size();
  std::vector<float> wbase((size_t)fmm::kMaxRank * 4, 0.0f);
  if (!shaped) fmm_realization_tables(d, 1, nullptr, nullptr, wbase.data());
  std::vector<float> wouter;
  if (q.depth >= 2) {
    const int no = 1 << (2 * (q.depth - 1));
    wouter.resize((size_t)pb.To * no);
    fmm_realization_tables(d, q.depth - 1, nullptr, nullptr, wouter.data());
  }
  // large-tile plans at depth 2 combine all T terms in one pass: the flattened w
  if (pb.split && q.depth == 2) {
    wfull.resize((size_t)T * 16);
    fmm_realization_tables(d, 2, nullptr, nullptr, wfull.data());
  }

  // device copy: [aoff][boff][aent][bent][winner][wouter][wfull][U][V]
  const size_t s_aoff = align256((T + 1) * sizeof(int32_t));
  const size_t s_boff = s_aoff;
  const size_t s_aent = align256(std::max<size_t>(1, aent.size()) * sizeof(fmm::CoefEntry));
  const size_t s_bent = align256(std::max<size_t>(1, bent.size()) * sizeof(fmm::CoefEntry));
  const size_t s_wi = align256(wbase.size() * sizeof(float));   // zero-padded to 8 x 4
  const size_t s_wo = align256(std::max<size_t>(1, wouter.size()) * sizeof(float));
  const size_t s_wf = align256(std::max<size_t>(1, wfull.size()) * sizeof(float));
  const size_t s_ud = align256(std::max<size_t>(1, U.size()) * sizeof(float));   // dense rows (the encoder at depths 2, 3)
  const size_t s_vd = align256(std::max<size_t>(1, V.size()) * sizeof(float));
  const size_t o_ud = s_aoff + s_boff + s_aent + s_bent + s_wi + s_wo + s_wf;
  const size_t tot = o_ud + s_ud + s_vd;
  std::vector<uint8_t> host(tot, 0);
  std::memcpy(host.data(), aoff.data(), (T + 1) * sizeof(int32_t));
  std::memcpy(host.data() + s_aoff, boff.data(), (T + 1) * sizeof(int32_t));
  if (!aent.empty()) std::memcpy(host.data() + s_aoff + s_boff, aent.data(), aent.size() * sizeof(fmm::CoefEntry));
  if (!bent.empty())
    std::memcpy(host.data() + s_aoff + s_boff + s_aent, bent.data(), bent.size() * sizeof(fmm::CoefEntry));
  std::memcpy(host.data() + s_aoff + s_boff + s_aent + s_bent, wbase.data(), wbase.size() * sizeof(float));
  if (!wouter.empty())
    std::memcpy(host.data() + s_aoff + s_boff + s_aent + s_bent + s_wi, wouter.data(),
                wouter.size() * sizeof(float));
  if (!U.empty()) std::memcpy(host.data() + o_ud, U.data(), U.size() * sizeof(float));
  if (!V.empty()) std::memcpy(host.data() + o_ud + s_ud, V.data(), V.size() * sizeof(float));
  if (!wfull.empty())
    std::memcpy(host.data() + s_aoff + s_boff + s_aent + s_bent + s_wi + s_wo, wfull.data(),
                wfull.size() * sizeof(float));

  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    delete p;
    return hip_status(hipErrorNoDevice);
  }
  if (!is_gfx950(dev)) {
    delete p;
    return FMM_ERR_DEVICE;
  }
  p->device = dev;
  void *dt = nullptr;
  int e = hipMalloc(&dt, tot);
  if (e == hipSuccess) e = hipMemcpy(dt, host.data(), tot, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    if (dt) (void)hipFree(dt);
    delete p;
    return hip_status(e);
  }
  p->dev_tables = dt;
  uint8_t *base = reinterpret_cast<uint8_t *>(dt);
  p->tab.a_off = reinterpret_cast<const int32_t *>(base);
  p->tab.b_off = reinterpret_cast<const int32_t *>(base + s_aoff);
  p->tab.a_ent = reinterpret_cast<const fmm::CoefEntry *>(base + s_aoff + s_boff);
  p->tab.b_ent = reinterpret_cast<const fmm::CoefEntry *>(base + s_aoff + s_boff + s_aent);
  p->tab.w_inner = reinterpret_cast<const float *>(base + s_aoff + s_boff + s_aent + s_bent);
  p->tab.w_outer = reinterpret_cast<const float *>(base + s_aoff + s_boff + s_aent + s_bent + s_wi);
  p->tab.w_full = reinterpret_cast<const float *>(base + s_aoff + s_boff + s_aent + s_bent + s_wi + s_wo);
  p->tab.u_dense = reinterpret_cast<const float *>(base + o_ud);
  p->tab.v_dense = reinterpret_cast<const float *>(base + o_ud + s_ud);
  *out = p;
  return FMM_OK;
}

int fmm_plan_workspace_size(const fmm_plan *p, size_t *bytes) {
  if (!p || !bytes) return FMM_ERR_ARG;
  *bytes = p->wl.total;
  return FMM_OK;
}

int fmm_operand_views(const fmm_plan *p, void *dWs, fmm_view *a, fmm_view *b) {
  if (!p) return FMM_ERR_ARG;
  uint8_t *ws = reinterpret_cast<uint8_t *>(dWs);
  const fmm::Problem &pb = p->pb;
  if (a) {
    a->codes = ws ? ws + p->wl.a_codes : nullptr;
    a->scales = ws ? ws + p->wl.a_scales : nullptr;
    a->batch = pb.batch; a->terms = pb.T; a->rows = pb.mp; a->kdim = pb.kp;
    a->kblocks = pb.kblocks; a->scale_bytes = pb.scale_bytes;
    a->code_layout = pb.layout;
  }
  if (b) {
    b->codes = ws ? ws + p->wl.b_codes : nullptr;
    b->scales = ws ? ws + p->wl.b_scales : nullptr;
    b->batch = pb.batch; b->terms = pb.T; b->rows = pb.np; b->kdim = pb.kp;
    b->kblocks = pb.kblocks; b->scale_bytes = pb.scale_bytes;
    b->code_layout = pb.layout;
  }
  return FMM_OK;
}

static int check_ws(const fmm_plan *p, const void *ws) {
  if (p->wl.total > 0 && !ws) return FMM_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % 256) return FMM_ERR_WORKSPACE;
  return FMM_OK;
}

int fmm_encode(const fmm_plan *p, const float *dA, const float *dB, void *dWs, void *stream) {
  if (!p) return FMM_ERR_ARG;
  const fmm::Problem &pb = p->pb;
  const bool empty = pb.batch == 0 || pb.M == 0 || pb.N == 0 || pb.K == 0;
  if (!empty && (!dA || !dB)) return FMM_ERR_ARG;
  if (!empty && ((reinterpret_cast<uintptr_t>(dA) | reinterpret_cast<uintptr_t>(dB)) % 16)) return FMM_ERR_ARG;
  int st = check_ws(p, dWs);
  if (st != FMM_OK) return st;
  return hip_status(fmm::launch_encode(pb, p->tab, dA, dB, reinterpret_cast<uint8_t *>(dWs), p->wl, stream));
}

static int check_multiply(const fmm_plan *p, const void *dWs, const float *dC) {
  if (!p) return FMM_ERR_ARG;
  const fmm::Problem &pb = p->pb;
  const bool empty = pb.batch == 0 || pb.M == 0 || pb.N == 0;
  if (!empty && !dC) return FMM_ERR_ARG;
  return check_ws(p, dWs);
}

int fmm_products(const fmm_plan *p, void *dWs, float *dC, void *stream) {
  int st = check_multiply(p, dWs, dC);
  if (st != FMM_OK) return st;
  return hip_status(fmm::launch_products(p->pb, p->tab, reinterpret_cast<const uint8_t *>(dWs), p->wl,
                                         dC, stream));
}

int fmm_combine(const fmm_plan *p, void *dWs, float *dC, void *stream) {
  int st = check_multiply(p, dWs, dC);
  if (st != FMM_OK) return st;
  return hip_status(fmm::launch_combine(p->pb, p->tab, reinterpret_cast<const uint8_t *>(dWs), p->wl,
                                        dC, stream));
}

int fmm_multiply(const fmm_plan *p, void *dWs, float *dC, void *stream) {
  int st = fmm_products(p, dWs, dC, stream);
  if (st != FMM_OK) return st;
  return fmm_combine(p, dWs, dC, stream);
}

int fmm_matmul(const fmm_plan *p, const float *dA, const float *dB, float *dC, void *dWs,
               void *stream) {
  int st = fmm_encode(p, dA, dB, dWs, stream);
  if (st != FMM_OK) return st;
  return fmm_multiply(p, dWs, dC, stream);
}

void fmm_plan_destroy(fmm_plan *p) {
  if (!p) return;
  if (p->dev_tables) (void)hipFree(p->dev_tables);
  delete p;
}

int fmm_reference_f64(int64_t batch, int64_t M, int64_t K, int64_t N, const float *dA,
                      const float *dB, double *dCref, void *stream) {
  if (batch < 0 || M < 0 || K < 0 || N < 0 || batch > 65535) return FMM_ERR_ARG;
  if (batch > 0 && M > 0 && N > 0 && (!dCref || (K > 0 && (!dA || !dB)))) return FMM_ERR_ARG;
  return hip_status(fmm::launch_reference_f64(batch, M, K, N, dA, dB, dCref, stream));
}

int fmm_error_stats_scratch_size(int64_t batch, int64_t M, int64_t N, size_t *bytes) {
  if (batch < 0 || M < 0 || N < 0 || !bytes) return FMM_ERR_ARG;
  *bytes = fmm::error_stats_scratch_bytes(batch, M, N);
  return FMM_OK;
}

int fmm_error_stats(int64_t batch, int64_t M, int64_t N, const float *dC, const double *dCref,
                    double *dOut, void *dScratch, size_t scratch_bytes, void *stream) {
  if (batch < 0 || M < 0 || N < 0 || batch > 65535) return FMM_ERR_ARG;
  if (batch == 0) return FMM_OK;
  if (!dOut || (M * N > 0 && (!dC || !dCref))) return FMM_ERR_ARG;
  if (!dScratch || scratch_bytes < fmm::error_stats_scratch_bytes(batch, M, N) ||
      reinterpret_cast<uintptr_t>(dScratch) % 8)
    return FMM_ERR_WORKSPACE;
  return hip_status(fmm::launch_error_stats(batch, M, N, dC, dCref, dOut, dScratch, stream));
}

int fmm_error_stats_noalloc(int64_t batch, int64_t M, int64_t N, const float *dC, const double *dCref,
                            double *dOut, void *stream) {
  if (batch < 0 || M < 0 || N < 0) return FMM_ERR_ARG;
  if (batch > fmm::kStaticErrorBatch) {
    g_detail = "fmm_error_stats_noalloc: batch " + std::to_string(batch) + " exceeds the static scratch (" +
               std::to_string(fmm::kStaticErrorBatch) + " products)";
    return FMM_ERR_WORKSPACE;
  }
  if (batch == 0) return FMM_OK;
  if (!dOut || (M * N > 0 && (!dC || !dCref))) return FMM_ERR_ARG;
  void *scratch = nullptr;
  const int e = fmm::static_error_scratch(&scratch);
  if (e != hipSuccess) return hip_status(e);
  return hip_status(fmm::launch_error_stats(batch, M, N, dC, dCref, dOut, scratch, stream));
}

int fmm_encode_noise_scratch_size(const fmm_plan *p, size_t *bytes) {
  if (!p || !bytes) return FMM_ERR_ARG;
  if (p->pb.depth > 2 || p->pb.shaped) return FMM_ERR_UNSUPPORTED;
  *bytes = fmm::encode_noise_scratch_bytes(p->pb);
  return FMM_OK;
}

int fmm_encode_noise(const fmm_plan *p, const float *dA, const float *dB, const void *dWs, double *dOut,
                     void *dScratch, size_t scratch_bytes, void *stream) {
  if (!p) return FMM_ERR_ARG;
  const fmm::Problem &pb = p->pb;
  if (pb.depth > 2 || pb.shaped) return FMM_ERR_UNSUPPORTED;
  if (pb.batch == 0) return FMM_OK;
  if (!dOut || !dWs || (pb.M * pb.K > 0 && !dA) || (pb.K * pb.N > 0 && !dB)) return FMM_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(dWs) % 256) return FMM_ERR_WORKSPACE;
  if (!dScratch || scratch_bytes < fmm::encode_noise_scratch_bytes(pb) || reinterpret_cast<uintptr_t>(dScratch) % 8)
    return FMM_ERR_WORKSPACE;
  return hip_status(fmm::launch_encode_noise(pb, p->tab, dA, dB, reinterpret_cast<const uint8_t *>(dWs), p->wl,
                                             dOut, dScratch, stream));
}

int fmm_cross_terms_scratch_size(const fmm_plan *p, size_t *bytes) {
  if (!p || !bytes) return FMM_ERR_ARG;
  if (p->pb.depth != 1 || p->pb.shaped) return FMM_ERR_UNSUPPORTED;
  *bytes = fmm::cross_terms_scratch_bytes(p->pb);
  return FMM_OK;
}

int fmm_cross_terms(const fmm_plan *p, const float *dA, const float *dB, const void *dWs, double *dOut,
                    void *dScratch, size_t scratch_bytes, void *stream) {
  if (!p) return FMM_ERR_ARG;
  const fmm::Problem &pb = p->pb;
  if (pb.depth != 1 || pb.shaped) return FMM_ERR_UNSUPPORTED;
  if (pb.batch == 0) return FMM_OK;
  if (!dOut || !dWs || (pb.M * pb.K > 0 && !dA) || (pb.K * pb.N > 0 && !dB)) return FMM_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(dWs) % 256) return FMM_ERR_WORKSPACE;
  if (!dScratch || scratch_bytes < fmm::cross_terms_scratch_bytes(pb) || reinterpret_cast<uintptr_t>(dScratch) % 256)
    return FMM_ERR_WORKSPACE;
  return hip_status(fmm::launch_cross_terms(pb, p->tab, dA, dB, reinterpret_cast<const uint8_t *>(dWs), p->wl,
                                            dOut, dScratch, stream));
}

int fmm_e4m3_quantize(const float *dIn, uint8_t *dOut, int64_t n, void *stream) {
  if (n < 0) return FMM_ERR_ARG;
  if (n == 0) return FMM_OK;
  if (!dIn || !dOut) return FMM_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(dIn) % 16 || reinterpret_cast<uintptr_t>(dOut) % 4) return FMM_ERR_ARG;
  return hip_status(fmm::launch_e4m3_quantize(dIn, dOut, n, stream));
}

int fmm_e4m3_quantize_pow2(const float *dIn, uint8_t *dOut, int64_t n, int32_t e, void *stream) {
  if (n < 0 || e < -126 || e > 127) return FMM_ERR_ARG;
  if (n == 0) return FMM_OK;
  if (!dIn || !dOut) return FMM_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(dIn) % 16 || reinterpret_cast<uintptr_t>(dOut) % 4) return FMM_ERR_ARG;
  return hip_status(fmm::launch_e4m3_quantize_pow2(dIn, dOut, n, e, stream));
}

}  // extern "C"
