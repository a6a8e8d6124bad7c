// api.hip -- the C ABI of libcold.so (declared in include/cold.h): model
// description checks, weight arena and workspace layout, and the launch
// sequence of one scoring call.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "cold.h"
#include "cold_internal.h"

using namespace cold;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct ArenaLayout {
  size_t tables, rows, magic, pairs, w1, b1, w2, b2, w1t, w2t, w1p, w2p, w1f, w2f;
  std::vector<size_t> w, b;
  size_t total;
};

struct WorkLayout {
  size_t err, U, zU, Uh, urow, X, E, actA, actB, sbuf, zbuf, partial, mask;
  size_t Xc, Wc, kept, rtiles, n_rtiles;   // compacted network input (see compact_input)
  size_t total;
};

}  // namespace

struct ProfSet {
  std::vector<hipEvent_t> ev;       // ev[i] precedes stage i; the last ends the call
  std::vector<const char *> names;
};

struct cold_model {
  cold_model_desc desc;
  std::vector<int32_t> widths;
  std::vector<int64_t> table_rows;
  std::vector<int32_t> cross_pairs;   // [n_cross][2] or empty
  int M, D_in, H, d, dtype, es, nus, hashed;
  bool literal_se;
  int max_hidden;
  ArenaLayout arena;
  unsigned char *arena_ptr = nullptr;
  bool loaded = false;
  std::vector<uint64_t> host_tables;  // staging for the arena's pointer table
  std::vector<uint64_t> host_magic;
  mutable std::mutex mu;
  std::string last_error;
  bool prof_on = false;
  std::vector<ProfSet> prof;        // one set of events per profiled call
  size_t prof_used = 0;
};

namespace {

int fail(cold_model *m, int status, const char *fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(cold_model *m, int status, const char *fmt, ...) {
  if (m) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    std::lock_guard<std::mutex> lk(m->mu);
    m->last_error = buf;
  }
  return status;
}

int hip_fail(cold_model *m, hipError_t e, const char *what) {
  return fail(m, COLD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// The top-k mask of the squeeze SE form without sequences runs as separate
// passes: gather with squeeze, SE of the rows, mask, reweighting in place.
// SE operands of the register-resident gather (squeeze form; its shape limits)
bool full_gather_model(const cold_model &m) {
  return !m.literal_se && gather_full_shape(m.M, m.H, m.d * m.es, m.desc.n_seq);
}

bool topk_split(const cold_model &m) {
  // the row-wise SE kernel holds M <= 256 groups and H <= 64 hidden units
  return m.desc.topk_k > 0 && !m.literal_se && m.desc.n_seq == 0 && m.M <= 256 && m.H <= 64;
}

// Top-k models whose first layer is a plain dense layer: each request's
// network input keeps only its k groups (in group order) and the first
// layer runs on them with the matching columns of its weights, which gives
// the masked input's products without the dropped groups' zeros (their
// products add nothing). Chosen by the model alone, for every batch size.
int kept_groups(const cold_model &m) { return m.desc.topk_k < m.M ? m.desc.topk_k : m.M; }

bool compact_input(const cold_model &m) {
  if (!topk_split(m) || kept_groups(m) >= m.M || m.dtype == kF32) return false;
  const int L = m.desc.n_layers;
  const bool fuse_tail = L >= 3 && tail_supported(m.dtype, m.widths[L - 3], m.widths[L - 2],
                                                  m.widths[L - 1], m.widths[L]);
  const int n_separate = fuse_tail ? L - 3 : L - 1;
  const bool dense_tail = fuse_tail && n_separate >= 1 &&
                          dense_tail_supported(m.dtype, 1, m.widths[n_separate], m.widths[n_separate - 1]);
  return n_separate - (dense_tail ? 1 : 0) >= 1 &&
         dense_grouped_supported(m.dtype, m.widths[1], kept_groups(m) * m.d);
}

ArenaLayout arena_layout(const cold_model &m) {
  ArenaLayout a;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  a.tables = take(sizeof(uint64_t) * m.M);
  a.rows = take(sizeof(int64_t) * m.M);
  a.magic = take(sizeof(uint64_t) * m.M);
  a.pairs = take(sizeof(int32_t) * m.cross_pairs.size());
  if (m.literal_se) {            // W [M][D_in], b [M]
    a.w1 = take(sizeof(float) * (size_t)m.M * m.D_in);
    a.b1 = take(sizeof(float) * m.M);
    a.w2 = take(0);
    a.b2 = take(0);
    a.w1t = take(0);
    a.w2t = take(0);
  } else {
    a.w1 = take(sizeof(float) * m.H * m.M);
    a.b1 = take(sizeof(float) * m.H);
    a.w2 = take(sizeof(float) * m.M * m.H);
    a.b2 = take(sizeof(float) * m.M);
    a.w1t = take(sizeof(float) * m.M * m.H);   // W1 as [M][H]
    a.w2t = take(sizeof(float) * m.H * m.M);   // W2 as [H][M]
  }
  size_t n1 = 0, n2 = 0;                        // the row-wise SE kernel's operands
  if (topk_split(m)) se_rows_packed_floats(m.M, m.H, &n1, &n2);
  a.w1p = take(sizeof(float) * n1);
  a.w2p = take(sizeof(float) * n2);
  a.w1f = take(full_gather_model(m) ? sizeof(float) * kSeFullFloats : 0);
  a.w2f = take(full_gather_model(m) ? sizeof(float) * kSeFullFloats : 0);
  const int L = m.desc.n_layers;
  for (int l = 0; l < L; ++l) {
    a.w.push_back(take((size_t)m.es * m.widths[l] * m.widths[l + 1]));
    a.b.push_back(take(sizeof(float) * m.widths[l + 1]));
  }
  a.total = off;
  return a;
}

WorkLayout work_layout(const cold_model &m, int64_t R, int64_t Q) {
  WorkLayout w;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += align_up(bytes); return o; };
  const bool topk = m.desc.topk_k > 0;
  const bool sbuf = topk || m.literal_se;
  w.err = take(sizeof(int32_t));
  w.U = take(sizeof(float) * (size_t)Q * m.nus * m.d);
  w.zU = take(sizeof(float) * (size_t)Q * m.nus);
  w.Uh = take((size_t)m.es * Q * m.desc.n_user * m.d);
  w.urow = take(sizeof(int32_t) * (size_t)Q * (m.desc.n_user > 0 ? m.desc.n_user : 1));
  w.X = take((size_t)m.es * R * m.D_in);
  w.E = take(m.literal_se ? sizeof(float) * (size_t)R * m.D_in : 0);
  w.actA = take((size_t)m.es * R * m.max_hidden);
  w.actB = take((size_t)m.es * R * m.max_hidden);
  w.sbuf = take(sbuf ? sizeof(float) * (size_t)R * m.M : 0);
  w.zbuf = take(topk_split(m) ? sizeof(float) * (size_t)R * m.M : 0);
  // per-request part sums of the mask, or the row-wise SE's 16-row tile sums
  const size_t parts = topk_split(m) ? (size_t)((R + 15) / 16) * m.M : (size_t)Q * kMaskParts * m.M;
  w.partial = take(topk ? sizeof(float) * parts : 0);
  w.mask = take(topk ? (size_t)Q * m.M : 0);
  const bool compact = compact_input(m);
  const size_t kin = compact ? (size_t)kept_groups(m) * m.d : 0;   // compacted input width
  w.Xc = take((size_t)m.es * R * kin);
  w.Wc = take(compact ? (size_t)m.es * Q * m.widths[1] * kin : 0);
  w.kept = take(compact ? sizeof(int32_t) * (size_t)Q * kept_groups(m) : 0);
  w.rtiles = take(compact ? sizeof(RowTile) * (size_t)row_tile_capacity(R, Q) : 0);
  w.n_rtiles = take(compact ? sizeof(int32_t) : 0);
  w.total = off;
  return w;
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

constexpr size_t kMaxProfiledCalls = 4096;

// Records the stage boundaries of one cold_score call when profiling is on.
struct StageMarks {
  cold_model *m;
  hipStream_t s;
  ProfSet *set = nullptr;
  size_t n = 0;
  StageMarks(cold_model *m_, hipStream_t s_, bool enabled) : m(m_), s(s_) {
    if (!enabled || !m->prof_on || m->prof_used >= kMaxProfiledCalls) return;
    if (m->prof_used == m->prof.size()) m->prof.emplace_back();
    set = &m->prof[m->prof_used++];
    set->names.clear();
  }
  hipError_t mark(const char *name) {  // name = NULL ends the call
    if (!set) return hipSuccess;
    if (n == set->ev.size()) {
      hipEvent_t e;
      hipError_t err = hipEventCreate(&e);
      if (err != hipSuccess) return err;
      set->ev.push_back(e);
    }
    if (name) set->names.push_back(name);
    return hipEventRecord(set->ev[n++], s);
  }
};

}  // namespace

extern "C" {

const char *cold_status_string(int status) {
  switch (status) {
    case COLD_OK: return "ok";
    case COLD_ERR_INVALID_ARG: return "invalid argument";
    case COLD_ERR_SHAPE: return "shape mismatch";
    case COLD_ERR_DTYPE: return "unsupported dtype or dimension";
    case COLD_ERR_NOT_LOADED: return "weights not loaded";
    case COLD_ERR_WORKSPACE: return "workspace or arena too small";
    case COLD_ERR_HIP: return "HIP runtime error";
    case COLD_ERR_ID_RANGE: return "id or offset out of range";
    default: return "unknown status";
  }
}

const char *cold_last_error(const cold_model *m) {
  if (!m) return "null model";
  std::lock_guard<std::mutex> lk(m->mu);
  return m->last_error.c_str();
}

int cold_create_model(const cold_model_desc *desc, cold_model **out) {
  if (!desc || !out) return COLD_ERR_INVALID_ARG;
  *out = nullptr;
  const cold_model_desc &D = *desc;
  if (D.n_user < 0 || D.n_seq < 0 || D.n_ad < 0 || D.n_cross < 0 || D.emb_dim <= 0 ||
      D.se_reduction < 1 || D.n_layers < 1 || !D.widths || !D.table_rows || D.topk_k < 0 ||
      (D.linear_log != 0 && D.linear_log != 1) ||
      (D.se_form != COLD_SE_SQUEEZE && D.se_form != COLD_SE_LITERAL))
    return COLD_ERR_INVALID_ARG;
  if (D.dtype != COLD_F32 && D.dtype != COLD_BF16 && D.dtype != COLD_F16) return COLD_ERR_DTYPE;
  if (D.id_kind != COLD_IDS_DIRECT_I32 && D.id_kind != COLD_IDS_HASHED_U64) return COLD_ERR_DTYPE;
  const int M = D.n_user + D.n_seq + D.n_ad + D.n_cross;
  if (M <= 0 || M > 1024) return COLD_ERR_SHAPE;
  const int es = D.dtype == COLD_F32 ? 4 : 2;
  const int epc = 16 / es;
  if ((D.emb_dim * es) % 16 != 0 || !is_pow2(D.emb_dim / epc) || D.emb_dim / epc > 64)
    return COLD_ERR_DTYPE;
  const int cpr = M * (D.emb_dim / epc);
  if (cpr > kGatherMaxChunksPerRow) return COLD_ERR_SHAPE;
  if (D.widths[0] != M * D.emb_dim) return COLD_ERR_SHAPE;
  const int n_out = D.widths[D.n_layers];
  if (n_out != 1 && n_out != 2) return COLD_ERR_SHAPE;
  int max_hidden = 0;
  for (int l = 1; l < D.n_layers; ++l) {
    if (D.widths[l] <= 0) return COLD_ERR_SHAPE;
    if (D.dtype != COLD_F32 && D.widths[l] % 8 != 0) return COLD_ERR_DTYPE;
    max_hidden = D.widths[l] > max_hidden ? D.widths[l] : max_hidden;
  }
  const int last_in = D.widths[D.n_layers - 1];
  if ((size_t)n_out * last_in * sizeof(float) > 64 * 1024) return COLD_ERR_SHAPE;
  for (int g = 0; g < M; ++g)
    if (D.table_rows[g] < 1 || D.table_rows[g] > 0x7FFFFFFF) return COLD_ERR_SHAPE;
  if (D.cross_pairs)
    for (int f = 0; f < D.n_cross; ++f)
      if (D.cross_pairs[2 * f] < 0 || D.cross_pairs[2 * f] >= D.n_user ||
          D.cross_pairs[2 * f + 1] < 0 || D.cross_pairs[2 * f + 1] >= D.n_ad)
        return COLD_ERR_SHAPE;

  cold_model *m = new (std::nothrow) cold_model();
  if (!m) return COLD_ERR_INVALID_ARG;
  m->desc = D;
  m->widths.assign(D.widths, D.widths + D.n_layers + 1);
  m->table_rows.assign(D.table_rows, D.table_rows + M);
  if (D.cross_pairs && D.n_cross > 0) m->cross_pairs.assign(D.cross_pairs, D.cross_pairs + 2 * D.n_cross);
  m->desc.widths = m->widths.data();
  m->desc.table_rows = m->table_rows.data();
  m->desc.cross_pairs = m->cross_pairs.empty() ? nullptr : m->cross_pairs.data();
  m->M = M;
  m->d = D.emb_dim;
  m->D_in = M * D.emb_dim;
  m->H = M / D.se_reduction > 0 ? M / D.se_reduction : 1;
  m->dtype = D.dtype;
  m->es = es;
  m->nus = D.n_user + D.n_seq;
  m->hashed = D.id_kind == COLD_IDS_HASHED_U64;
  m->literal_se = D.se_form == COLD_SE_LITERAL;
  m->max_hidden = max_hidden;
  m->arena = arena_layout(*m);
  m->host_tables.assign(M, 0);
  m->host_magic.resize(M);
  for (int g = 0; g < M; ++g) m->host_magic[g] = ~0ull / (uint64_t)m->table_rows[g];
  *out = m;
  return COLD_OK;
}

static void destroy_events(cold_model *m) {
  for (ProfSet &p : m->prof)
    for (hipEvent_t e : p.ev) (void)hipEventDestroy(e);
  m->prof.clear();
  m->prof_used = 0;
}

void cold_destroy_model(cold_model *m) {
  if (!m) return;
  destroy_events(m);
  delete m;
}

int cold_profile_enable(cold_model *m, int32_t enable) {
  if (!m) return COLD_ERR_INVALID_ARG;
  m->prof_on = enable != 0;
  if (!m->prof_on) destroy_events(m);
  m->prof_used = 0;
  return COLD_OK;
}

int cold_profile_read(cold_model *m, int32_t max_stages, char (*names)[32], float *total_ms,
                      int32_t *n_stages, int32_t *n_calls) {
  if (!m || max_stages < 0 || (!total_ms && max_stages > 0) || !n_stages || !n_calls)
    return COLD_ERR_INVALID_ARG;
  *n_stages = 0;
  *n_calls = (int32_t)m->prof_used;
  for (int i = 0; i < max_stages; ++i) total_ms[i] = 0.0f;
  for (size_t c = 0; c < m->prof_used; ++c) {
    ProfSet &p = m->prof[c];
    const int ns = (int)p.names.size();
    if (c == 0) *n_stages = ns;
    else if (ns != *n_stages) return fail(m, COLD_ERR_INVALID_ARG, "profiled calls differ in stages");
    hipError_t e = hipEventSynchronize(p.ev[ns]);
    if (e != hipSuccess) return hip_fail(m, e, "cold_profile_read: synchronize");
    for (int i = 0; i < ns && i < max_stages; ++i) {
      float ms = 0.0f;
      if ((e = hipEventElapsedTime(&ms, p.ev[i], p.ev[i + 1])) != hipSuccess)
        return hip_fail(m, e, "cold_profile_read: elapsed");
      total_ms[i] += ms;
      if (names && c == 0) {
        std::strncpy(names[i], p.names[i], 31);
        names[i][31] = 0;
      }
    }
  }
  m->prof_used = 0;
  return COLD_OK;
}

size_t cold_weight_arena_bytes(const cold_model *m) { return m ? m->arena.total : 0; }

size_t cold_workspace_bytes(const cold_model *m, int64_t max_rows, int64_t max_requests) {
  if (!m || max_rows < 0 || max_requests < 0) return 0;
  return work_layout(*m, max_rows, max_requests).total;
}

int cold_load_weights(cold_model *m, const cold_weights *w, void *arena, size_t arena_bytes,
                      void *stream) {
  if (!m) return COLD_ERR_INVALID_ARG;
  if (!w || !arena || !w->tables || !w->se_w1 || !w->se_b1 ||
      (!m->literal_se && (!w->se_w2 || !w->se_b2)) || !w->mlp_w || !w->mlp_b)
    return fail(m, COLD_ERR_INVALID_ARG, "cold_load_weights: null pointer");
  if (reinterpret_cast<uintptr_t>(arena) % kAlign)
    return fail(m, COLD_ERR_INVALID_ARG, "arena must be %zu-byte aligned", kAlign);
  if (arena_bytes < m->arena.total)
    return fail(m, COLD_ERR_WORKSPACE, "arena has %zu bytes, needs %zu", arena_bytes, m->arena.total);
  for (int g = 0; g < m->M; ++g) {
    if (!w->tables[g] || reinterpret_cast<uintptr_t>(w->tables[g]) % 16)
      return fail(m, COLD_ERR_INVALID_ARG, "table %d is null or not 16-byte aligned", g);
    m->host_tables[g] = reinterpret_cast<uint64_t>(w->tables[g]);
  }
  const int L = m->desc.n_layers;
  for (int l = 0; l < L; ++l)
    if (!w->mlp_w[l] || !w->mlp_b[l]) return fail(m, COLD_ERR_INVALID_ARG, "layer %d weights null", l);

  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char *A = static_cast<unsigned char *>(arena);
  const ArenaLayout &al = m->arena;
  struct Copy { size_t off; const void *src; size_t bytes; hipMemcpyKind kind; };
  std::vector<Copy> copies = {
      {al.tables, m->host_tables.data(), sizeof(uint64_t) * m->M, hipMemcpyHostToDevice},
      {al.rows, m->table_rows.data(), sizeof(int64_t) * m->M, hipMemcpyHostToDevice},
      {al.magic, m->host_magic.data(), sizeof(uint64_t) * m->M, hipMemcpyHostToDevice},
      {al.pairs, m->cross_pairs.data(), sizeof(int32_t) * m->cross_pairs.size(), hipMemcpyHostToDevice},
      {al.w1, w->se_w1, sizeof(float) * (m->literal_se ? (size_t)m->M * m->D_in : (size_t)m->H * m->M),
       hipMemcpyDeviceToDevice},
      {al.b1, w->se_b1, sizeof(float) * (m->literal_se ? m->M : m->H), hipMemcpyDeviceToDevice},
      {al.w2, w->se_w2, m->literal_se ? 0 : sizeof(float) * m->M * m->H, hipMemcpyDeviceToDevice},
      {al.b2, w->se_b2, m->literal_se ? 0 : sizeof(float) * m->M, hipMemcpyDeviceToDevice}};
  // the fused tail's two hidden layers are stored fragment-major; every
  // other weight matrix is copied as given
  const bool fuse_tail = L >= 3 && tail_supported(m->dtype, m->widths[L - 3], m->widths[L - 2],
                                                  m->widths[L - 1], m->widths[L]);
  auto packed = [&](int l) { return fuse_tail && (l == L - 3 || l == L - 2); };
  for (int l = 0; l < L; ++l) {
    if (!packed(l))
      copies.push_back({al.w[l], w->mlp_w[l], (size_t)m->es * m->widths[l] * m->widths[l + 1],
                        hipMemcpyDeviceToDevice});
    copies.push_back({al.b[l], w->mlp_b[l], sizeof(float) * m->widths[l + 1], hipMemcpyDeviceToDevice});
  }
  for (const Copy &c : copies) {
    if (c.bytes == 0) continue;
    hipError_t e = hipMemcpyAsync(A + c.off, c.src, c.bytes, c.kind, s);
    if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: copy");
  }
  if (!m->literal_se) {
    // transposed SE weights for the gathers that read them from global memory
    hipError_t e = launch_transpose_f32(reinterpret_cast<const float *>(A + al.w1),
                                        reinterpret_cast<float *>(A + al.w1t), m->H, m->M, s);
    if (e == hipSuccess)
      e = launch_transpose_f32(reinterpret_cast<const float *>(A + al.w2),
                               reinterpret_cast<float *>(A + al.w2t), m->M, m->H, s);
    if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: transpose");
  }
  if (topk_split(*m)) {
    hipError_t e = launch_pack_se_rows(reinterpret_cast<const float *>(A + al.w1),
                                       reinterpret_cast<const float *>(A + al.w2), m->M, m->H,
                                       reinterpret_cast<float *>(A + al.w1p),
                                       reinterpret_cast<float *>(A + al.w2p), s);
    if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: SE pack");
  }
  if (full_gather_model(*m)) {
    hipError_t e = launch_pack_se_full(reinterpret_cast<const float *>(A + al.w1),
                                       reinterpret_cast<const float *>(A + al.w2), m->M, m->H,
                                       reinterpret_cast<float *>(A + al.w1f),
                                       reinterpret_cast<float *>(A + al.w2f), s);
    if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: SE pack");
  }
  for (int l = 0; l < L; ++l)
    if (packed(l)) {
      hipError_t e = launch_pack_frag(w->mlp_w[l], A + al.w[l], m->widths[l + 1], m->widths[l], s);
      if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: pack");
    }
  hipError_t e = hipStreamSynchronize(s);  // host staging must outlive the copies
  if (e != hipSuccess) return hip_fail(m, e, "cold_load_weights: synchronize");
  m->arena_ptr = A;
  m->loaded = true;
  return COLD_OK;
}

}  // extern "C"

namespace {

// Host-side checks of a scoring call that do not involve the workspace.
// Returns COLD_OK, a negative status (recorded on the model), or 1 for a
// valid empty batch (nothing to do).
int check_call(cold_model *m, const cold_batch *b, const float *scores, int32_t flags,
               const char *who) {
  if (!m) return COLD_ERR_INVALID_ARG;
  if (!b) return fail(m, COLD_ERR_INVALID_ARG, "%s: null batch", who);
  if (flags & ~COLD_SCORE_VALIDATE) return fail(m, COLD_ERR_INVALID_ARG, "unknown flags 0x%x", flags);
  if (!m->loaded) return fail(m, COLD_ERR_NOT_LOADED, "%s before cold_load_weights", who);
  const int64_t Q = b->n_requests, R = b->n_rows;
  if (Q < 0 || R < 0 || b->n_seq_ids < 0) return fail(m, COLD_ERR_INVALID_ARG, "negative size");
  if (Q == 0 && R > 0) return fail(m, COLD_ERR_SHAPE, "rows without requests");
  if (R > 0x7FFFFFFFll * 16 || Q > 0x7FFFFFFF) return fail(m, COLD_ERR_SHAPE, "batch too large");
  if (Q == 0 || R == 0) return 1;
  const cold_model_desc &D = m->desc;
  if (!b->req_off || !scores ||
      (D.n_user > 0 && !b->user_ids) || (D.n_ad > 0 && !b->ad_ids) ||
      (D.n_cross > 0 && !D.cross_pairs && !b->cross_ids) || (D.n_seq > 0 && !b->seq_off) ||
      (D.n_seq > 0 && b->n_seq_ids > 0 && !b->seq_ids))
    return fail(m, COLD_ERR_INVALID_ARG, "%s: null pointer", who);
  return COLD_OK;
}

// The launch sequence of one scoring call on a checked batch, with the
// workspace regions at W (work_layout(R, Q) bytes, 256-byte aligned).  With
// profile, stage events are recorded when the model's profiling is on.
int score_launch(cold_model *m, const cold_batch *b, unsigned char *W, float *scores,
                 float *importance, uint8_t *group_mask, int32_t *rows_out, void *x_out,
                 int32_t flags, hipStream_t s, bool profile) {
  const int64_t Q = b->n_requests, R = b->n_rows;
  const cold_model_desc &D = m->desc;
  const WorkLayout wl = work_layout(*m, R, Q);
  unsigned char *A = m->arena_ptr;
  const ArenaLayout &al = m->arena;
  const bool topk = D.topk_k > 0;

  GatherArgs g{};
  g.M = m->M; g.n_user = D.n_user; g.n_seq = D.n_seq; g.n_ad = D.n_ad; g.n_cross = D.n_cross;
  g.d = m->d; g.H = m->H;
  g.R = R; g.Q = Q; g.n_seq_ids = b->n_seq_ids;
  g.req_off = b->req_off; g.user_ids = b->user_ids; g.ad_ids = b->ad_ids; g.cross_ids = b->cross_ids;
  g.seq_off = b->seq_off; g.seq_ids = b->seq_ids;
  g.tables = reinterpret_cast<const void *const *>(A + al.tables);
  g.table_rows = reinterpret_cast<const int64_t *>(A + al.rows);
  g.table_magic = reinterpret_cast<const uint64_t *>(A + al.magic);
  g.cross_pairs = D.cross_pairs ? reinterpret_cast<const int32_t *>(A + al.pairs) : nullptr;
  g.w1 = reinterpret_cast<const float *>(A + al.w1);
  g.b1 = reinterpret_cast<const float *>(A + al.b1);
  g.w2 = reinterpret_cast<const float *>(A + al.w2);
  g.b2 = reinterpret_cast<const float *>(A + al.b2);
  g.w1t = reinterpret_cast<const float *>(A + al.w1t);
  g.w2t = reinterpret_cast<const float *>(A + al.w2t);
  g.w1f = full_gather_model(*m) ? reinterpret_cast<const float *>(A + al.w1f) : nullptr;
  g.w2f = full_gather_model(*m) ? reinterpret_cast<const float *>(A + al.w2f) : nullptr;
  g.U = reinterpret_cast<float *>(W + wl.U);
  g.zU = reinterpret_cast<float *>(W + wl.zU);
  g.Uh = W + wl.Uh;
  g.urow = reinterpret_cast<int32_t *>(W + wl.urow);
  g.X = W + wl.X;
  g.rows_out = rows_out;
  g.err = reinterpret_cast<int32_t *>(W + wl.err);

  hipError_t e;
  const bool validate = flags & COLD_SCORE_VALIDATE;
  StageMarks marks(m, s, profile);
  static const char *kDenseNames[] = {"dense0", "dense1", "dense2", "dense3", "dense4", "dense5",
                                      "dense6", "dense7", "dense8", "dense9", "dense10", "dense11"};
  if (validate && (e = launch_clear_flag(g.err, s)) != hipSuccess) return hip_fail(m, e, "clear");
  // the one-pass SE (no top-k) of small models runs on the register-resident gather
  const bool full = !m->literal_se && !topk && gather_full_supported(m->dtype, g);
  // top-k models with a compacted network input (the first layer per request)
  const bool compact = compact_input(*m);
  float *sb_compact = compact ? (importance ? importance : reinterpret_cast<float *>(W + wl.sbuf)) : nullptr;
  if (user_pool_needed(m->dtype, g)) {   // per-request user rows and pooled sequences
    if ((e = marks.mark("user_pool")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_user_pool(m->dtype, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "user_pool launch");
  }
  if (m->literal_se) {
    // Eq. 2 as printed: the concatenated embedding (fp32), one dense layer
    // with a sigmoid to the M weights, then the reweighting pass
    float *sb = importance ? importance : reinterpret_cast<float *>(W + wl.sbuf);
    g.X = W + wl.E;
    if ((e = marks.mark("gather_raw")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_gather_se(m->dtype, kRawOut, false, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "gather (raw) launch");
    if ((e = marks.mark("se_dense")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_dense_f32(reinterpret_cast<const float *>(W + wl.E), g.w1, g.b1, sb, R, m->M,
                              m->D_in, 2, s)) != hipSuccess)
      return hip_fail(m, e, "SE layer launch");
    g.mask = nullptr;
    if (topk) {
      uint8_t *mask = W + wl.mask;
      if ((e = marks.mark("group_mask")) != hipSuccess) return hip_fail(m, e, "profile event");
      if ((e = launch_group_mask(sb, b->req_off, Q, R, m->M, D.topk_k,
                                 reinterpret_cast<float *>(W + wl.partial), kMaskParts, mask,
                                 group_mask, s)) != hipSuccess)
        return hip_fail(m, e, "group_mask launch");
      g.mask = mask;
    }
    g.s_buf = sb;
    g.X = W + wl.X;
    g.rows_out = nullptr;  // written by the first pass
    if ((e = marks.mark("gather_apply")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_gather_se(m->dtype, kApplyWeights, D.linear_log, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "gather_se (apply) launch");
  } else if (!topk) {
    g.s_buf = importance;
    if ((e = marks.mark("gather_se")) != hipSuccess) return hip_fail(m, e, "profile event");
    e = full ? launch_gather_full(m->dtype, D.linear_log, m->hashed, g, s)
             : launch_gather_se(m->dtype, kFull, D.linear_log, m->hashed, g, s);
    if (e != hipSuccess) return hip_fail(m, e, "gather_se launch");
  } else if (topk_split(*m)) {
    // gather with squeeze (rows kept exact in the input's place), SE of the
    // rows on the matrix cores with their 16-row tile sums, the per-request
    // mask in one launch, reweighting in place
    float *sb = importance ? importance : reinterpret_cast<float *>(W + wl.sbuf);
    uint8_t *mask = W + wl.mask;
    g.s_buf = nullptr;
    g.z_out = reinterpret_cast<float *>(W + wl.zbuf);
    if ((e = marks.mark("gather_sq")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_gather_se(m->dtype, kSqueezeRaw, false, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "gather_se (squeeze) launch");
    if ((e = marks.mark("se_rows")) != hipSuccess) return hip_fail(m, e, "profile event");
    float *tpart = reinterpret_cast<float *>(W + wl.partial);
    if ((e = launch_se_rows(g.z_out, sb, R, m->M, m->H, reinterpret_cast<const float *>(A + al.w1p), g.b1,
                              reinterpret_cast<const float *>(A + al.w2p), g.b2, tpart, s)) != hipSuccess)
      return hip_fail(m, e, "se_rows launch");
    if ((e = marks.mark("group_mask")) != hipSuccess) return hip_fail(m, e, "profile event");
    int32_t *kept = compact ? reinterpret_cast<int32_t *>(W + wl.kept) : nullptr;
    if ((e = launch_group_mask_tiles(sb, tpart, b->req_off, Q, R, m->M, D.topk_k, mask, group_mask,
                                     kept, s)) != hipSuccess)
      return hip_fail(m, e, "group_mask launch");
    if (compact) {
      // the rows' kept groups reweighted into the compacted input, every
      // request's columns of the first layer's weights and the layer's row
      // tiles, in one launch
      if ((e = marks.mark("apply_compact")) != hipSuccess) return hip_fail(m, e, "profile event");
      if ((e = launch_apply_compact(m->dtype, D.linear_log, W + wl.X, W + wl.Xc, sb, kept, b->req_off,
                                    Q, R, m->M, kept_groups(*m), m->d, A + al.w[0], m->widths[1],
                                    W + wl.Wc, reinterpret_cast<RowTile *>(W + wl.rtiles),
                                    reinterpret_cast<int32_t *>(W + wl.n_rtiles), s)) != hipSuccess)
        return hip_fail(m, e, "apply launch");
    } else {
      if ((e = marks.mark("apply")) != hipSuccess) return hip_fail(m, e, "profile event");
      if ((e = launch_apply_weights(m->dtype, D.linear_log, W + wl.X, sb, mask, b->req_off, Q, R, m->M,
                                    m->d, s)) != hipSuccess)
        return hip_fail(m, e, "apply launch");
    }
  } else {
    float *sb = importance ? importance : reinterpret_cast<float *>(W + wl.sbuf);
    uint8_t *mask = W + wl.mask;
    g.s_buf = sb;
    if ((e = marks.mark("se_weights")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_gather_se(m->dtype, kWeightsOnly, false, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "gather_se (weights) launch");
    if ((e = marks.mark("group_mask")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_group_mask(sb, b->req_off, Q, R, m->M, D.topk_k,
                               reinterpret_cast<float *>(W + wl.partial), kMaskParts, mask,
                               group_mask, s)) != hipSuccess)
      return hip_fail(m, e, "group_mask launch");
    g.mask = mask;
    g.rows_out = nullptr;  // written by the first pass
    if ((e = marks.mark("gather_apply")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_gather_se(m->dtype, kApplyWeights, D.linear_log, m->hashed, g, s)) != hipSuccess)
      return hip_fail(m, e, "gather_se (apply) launch");
  }
  if (x_out) {   // debug copy of the network input
    if ((e = hipMemcpyAsync(x_out, W + wl.X, (size_t)m->es * R * m->D_in, hipMemcpyDeviceToDevice,
                            s)) != hipSuccess)
      return hip_fail(m, e, "network input copy");
    // the compacted form keeps the gathered rows in X: the masked input
    // (dropped groups zero) is formed in the copy
    if (compact && (e = launch_apply_weights(m->dtype, D.linear_log, x_out, sb_compact, W + wl.mask,
                                             b->req_off, Q, R, m->M, m->d, s)) != hipSuccess)
      return hip_fail(m, e, "network input copy (masked)");
  }
  // network: hidden layers ping-pong between two activation buffers; the
  // last two hidden layers and the head run fused when their widths allow
  const int L = D.n_layers;
  const bool fuse_tail = L >= 3 && tail_supported(m->dtype, m->widths[L - 3], m->widths[L - 2],
                                                  m->widths[L - 1], m->widths[L]);
  const int n_separate = fuse_tail ? L - 3 : L - 1;
  // the last separate layer runs in the tail's kernel when it is 256 wide
  // with K in 64-deep steps, for every batch size (the choice depends on the
  // model alone, so a score does not depend on the batch it is scored in)
  const bool dense_tail = fuse_tail && n_separate >= 1 &&
                          dense_tail_supported(m->dtype, R, m->widths[n_separate],
                                               m->widths[n_separate - 1]);
  const void *in = W + wl.X;
  unsigned char *bufs[2] = {W + wl.actA, W + wl.actB};
  for (int l = 0; l < n_separate - (dense_tail ? 1 : 0); ++l) {
    void *outp = bufs[l & 1];
    if ((e = marks.mark(l < 12 ? kDenseNames[l] : "dense")) != hipSuccess)
      return hip_fail(m, e, "profile event");
    if (l == 0 && compact)
      e = launch_dense_relu_grouped(m->dtype, W + wl.Xc, W + wl.Wc,
                                    reinterpret_cast<const float *>(A + al.b[0]), outp, R, Q,
                                    m->widths[1], kept_groups(*m) * m->d,
                                    reinterpret_cast<RowTile *>(W + wl.rtiles),
                                    reinterpret_cast<int32_t *>(W + wl.n_rtiles), s);
    else
      e = launch_dense_relu(m->dtype, in, A + al.w[l], reinterpret_cast<const float *>(A + al.b[l]),
                            outp, R, m->widths[l + 1], m->widths[l], s);
    if (e != hipSuccess) return hip_fail(m, e, "dense layer launch");
    in = outp;
  }
  if (dense_tail) {
    const int l = n_separate - 1;
    if ((e = marks.mark("dense_tail")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_dense_tail(m->dtype, in, A + al.w[l], reinterpret_cast<const float *>(A + al.b[l]),
                               m->widths[l + 1], m->widths[l], A + al.w[L - 3],
                               reinterpret_cast<const float *>(A + al.b[L - 3]), A + al.w[L - 2],
                               reinterpret_cast<const float *>(A + al.b[L - 2]), A + al.w[L - 1],
                               reinterpret_cast<const float *>(A + al.b[L - 1]), m->widths[L],
                               scores, R, s)) != hipSuccess)
      return hip_fail(m, e, "dense + tail launch");
  } else if (fuse_tail) {
    if ((e = marks.mark("tail")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_mlp_tail(m->dtype, in, A + al.w[L - 3], reinterpret_cast<const float *>(A + al.b[L - 3]),
                             A + al.w[L - 2], reinterpret_cast<const float *>(A + al.b[L - 2]),
                             A + al.w[L - 1], reinterpret_cast<const float *>(A + al.b[L - 1]),
                             m->widths[L], scores, R, s)) != hipSuccess)
      return hip_fail(m, e, "tail launch");
  } else {
    if ((e = marks.mark("head")) != hipSuccess) return hip_fail(m, e, "profile event");
    if ((e = launch_head(m->dtype, in, A + al.w[L - 1], reinterpret_cast<const float *>(A + al.b[L - 1]),
                         scores, R, m->widths[L - 1], m->widths[L], s)) != hipSuccess)
      return hip_fail(m, e, "head launch");
  }
  if ((e = marks.mark(nullptr)) != hipSuccess) return hip_fail(m, e, "profile event");
  if (validate) {
    int32_t flag = 0;
    if ((e = hipMemcpyAsync(&flag, g.err, sizeof flag, hipMemcpyDeviceToHost, s)) != hipSuccess)
      return hip_fail(m, e, "flag readback");
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(m, e, "synchronize");
    if (flag) return fail(m, COLD_ERR_ID_RANGE, "out-of-range %s%s", (flag & 1) ? "ids " : "",
                          (flag & 2) ? "offsets" : "");
  }
  return COLD_OK;
}

}  // namespace

extern "C" {

int cold_score(cold_model *m, const cold_batch *b, void *workspace, size_t ws_bytes, float *scores,
               float *importance, uint8_t *group_mask, int32_t *rows_out, void *x_out,
               int32_t flags, void *stream) {
  const int st = check_call(m, b, scores, flags, "cold_score");
  if (st != COLD_OK) return st == 1 ? COLD_OK : st;
  if (!workspace) return fail(m, COLD_ERR_INVALID_ARG, "cold_score: null pointer");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(m, COLD_ERR_INVALID_ARG, "workspace must be %zu-byte aligned", kAlign);
  const size_t need = work_layout(*m, b->n_rows, b->n_requests).total;
  if (ws_bytes < need)
    return fail(m, COLD_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, need);
  return score_launch(m, b, static_cast<unsigned char *>(workspace), scores, importance, group_mask,
                      rows_out, x_out, flags, static_cast<hipStream_t>(stream), true);
}

}  // extern "C"

// ------------------------------------------------- scoring without allocation
// The workspace of cold_score_noalloc: a device array the library holds,
// one copy per GPU it runs on, until the process ends.  In host code this
// name is not a device address; hipGetSymbolAddress gives each device's copy.
static __device__ __align__(256) unsigned char scratch[COLD_NOALLOC_WORKSPACE_BYTES];

static_assert(COLD_NOALLOC_WORKSPACE_BYTES % 256 == 0, "workspace regions are 256-byte aligned");

namespace {

// Device address of `scratch` on device dev (the current device), looked up
// once per device and kept.
hipError_t scratch_address(int dev, unsigned char **out) {
  static std::mutex mu;
  static std::vector<std::pair<int, unsigned char *>> known;
  std::lock_guard<std::mutex> lk(mu);
  for (const auto &e : known)
    if (e.first == dev) {
      *out = e.second;
      return hipSuccess;
    }
  void *p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!p) return hipErrorInvalidSymbol;
  known.emplace_back(dev, static_cast<unsigned char *>(p));
  *out = static_cast<unsigned char *>(p);
  return hipSuccess;
}

}  // namespace

extern "C" {

int cold_score_noalloc(cold_model *m, const cold_batch *b, float *scores, float *importance,
                       uint8_t *group_mask, int32_t *rows_out, void *x_out, int32_t flags,
                       void *stream) {
  const int st = check_call(m, b, scores, flags, "cold_score_noalloc");
  if (st != COLD_OK) return st == 1 ? COLD_OK : st;
  const size_t need = work_layout(*m, b->n_rows, b->n_requests).total;
  if (need > COLD_NOALLOC_WORKSPACE_BYTES)
    return fail(m, COLD_ERR_WORKSPACE,
                "cold_score_noalloc: the batch needs %zu bytes of workspace, more than the "
                "library's %llu-byte array; score it with cold_score and a workspace",
                need, (unsigned long long)COLD_NOALLOC_WORKSPACE_BYTES);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int cur = -1, dev = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return hip_fail(m, e, "cold_score_noalloc: current device");
  dev = cur;
  if (s && (e = hipStreamGetDevice(s, &dev)) != hipSuccess)
    return hip_fail(m, e, "cold_score_noalloc: stream device");
  if (dev != cur)
    return fail(m, COLD_ERR_INVALID_ARG,
                "cold_score_noalloc: the stream is on device %d, the current device is %d", dev,
                cur);
  unsigned char *W = nullptr;
  if ((e = scratch_address(dev, &W)) != hipSuccess)
    return hip_fail(m, e, "cold_score_noalloc: workspace address");
  return score_launch(m, b, W, scores, importance, group_mask, rows_out, x_out, flags, s, false);
}

}  // extern "C"
