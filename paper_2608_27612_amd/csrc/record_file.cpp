// Record files: an emr_sink that appends every delivery of a streamed discovery to a file, so a
// deep run's output is bounded by the disk and not by host memory (Section 6 streams depth-13
// substrates from disk), and a run that stopped (a refused delivery, a full disk, a killed
// process) resumes from the file's last whole delivery.
//
// Layout (little-endian): a 32-byte header {char magic[8] = "EMRRECv1", int64 n_pairs, int64 0,
// int64 0}, then one block per delivery in cursor order: {int64 pair, int64 chunk, int64 n}
// followed by uint32 parent[n] and float w4[4 n]. Host only.
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <cerrno>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/emr.h"

namespace emr {
emr_status set_error(emr_status st, const std::string& msg);
}

struct emr_record_file {
  FILE* f = nullptr;
  int64_t n_pairs = 0;
  int64_t next = 0;     // cursor after the last whole delivery in the file
  int64_t records = 0;  // records in the file
  // EMR_E_IO after a failed write, EMR_E_INVAL after a refused delivery; later deliveries are
  // refused and the close call returns it
  emr_status failed = EMR_OK;
  std::string msg;
  std::vector<char> buf;
};

namespace {

constexpr char kMagic[8] = {'E', 'M', 'R', 'R', 'E', 'C', 'v', '1'};
constexpr int64_t kHeaderBytes = 32;
constexpr int64_t kBlockHeaderBytes = 24;
constexpr int64_t kRecordBytes = 20;
constexpr int64_t kDefaultBuffer = 8 << 20;
constexpr int64_t kMaxBuffer = int64_t(1) << 30;

emr_status failf(emr_status st, const char* fmt, ...) {
  char b[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(b, sizeof b, fmt, ap);
  va_end(ap);
  return emr::set_error(st, b);
}

bool read_exact(FILE* f, void* p, size_t n) { return std::fread(p, 1, n, f) == n; }

// Scans an existing file's blocks, keeping every whole one: returns the byte length of the
// whole blocks (a trailing partial block is left out), the cursor after the last one and the
// records they hold. EMR_E_INVAL when a block header is not one this sink could have written.
emr_status scan(FILE* f, int64_t size, int64_t n_pairs, int64_t* end, int64_t* next,
                int64_t* records) {
  int64_t pos = kHeaderBytes, cur = -1, recs = 0;
  while (pos + kBlockHeaderBytes <= size) {
    int64_t h[3];
    if (::fseeko(f, (off_t)pos, SEEK_SET) != 0 || !read_exact(f, h, sizeof h))
      return failf(EMR_E_IO, "record file: cannot read the block at offset %lld", (long long)pos);
    const int64_t pair = h[0], chunk = h[1], n = h[2];
    if (pair < 0 || pair >= n_pairs || chunk < 0 || chunk > (INT64_MAX - pair) / n_pairs ||
        n < 1 || n > (INT64_MAX - pos) / kRecordBytes)
      return failf(EMR_E_INVAL, "record file: malformed block at offset %lld (pair %lld, chunk "
                   "%lld, %lld records)", (long long)pos, (long long)pair, (long long)chunk,
                   (long long)n);
    const int64_t c = chunk * n_pairs + pair;
    if (c <= cur)
      return failf(EMR_E_INVAL, "record file: block at offset %lld has cursor %lld after %lld",
                   (long long)pos, (long long)c, (long long)cur);
    const int64_t block = kBlockHeaderBytes + n * kRecordBytes;
    if (pos + block > size) break;  // partial: the writer stopped inside this block
    pos += block;
    cur = c;
    recs += n;
  }
  *end = pos;
  *next = cur + 1;
  *records = recs;
  return EMR_OK;
}

emr_status open_file(const char* path, int64_t n_pairs, int32_t resume, int64_t buffer_bytes,
                     emr_record_file** out, int64_t* cursor) {
  if (!out) return failf(EMR_E_INVAL, "record file: out is NULL");
  *out = nullptr;
  if (!path || !*path) return failf(EMR_E_INVAL, "record file: empty path");
  if (n_pairs < 1) return failf(EMR_E_INVAL, "record file: n_pairs %lld < 1", (long long)n_pairs);
  if (resume != 0 && resume != 1) return failf(EMR_E_INVAL, "record file: resume must be 0 or 1");
  if (buffer_bytes < 0 || buffer_bytes > kMaxBuffer)
    return failf(EMR_E_INVAL, "record file: buffer_bytes %lld outside [0, 2^30]",
                 (long long)buffer_bytes);
  auto* F = new emr_record_file;
  F->n_pairs = n_pairs;
  struct stat sb;
  const bool exists = ::stat(path, &sb) == 0;
  if (resume && exists) {
    F->f = std::fopen(path, "r+b");
    if (!F->f) {
      delete F;
      return failf(EMR_E_IO, "record file: cannot open %s: %s", path, std::strerror(errno));
    }
    char magic[8];
    int64_t h[3];
    const int64_t size = (int64_t)sb.st_size;
    if (size < kHeaderBytes || !read_exact(F->f, magic, 8) || !read_exact(F->f, h, sizeof h) ||
        std::memcmp(magic, kMagic, 8) != 0) {
      std::fclose(F->f);
      delete F;
      return failf(EMR_E_INVAL, "record file: %s is not a record file", path);
    }
    if (h[0] != n_pairs) {
      std::fclose(F->f);
      delete F;
      return failf(EMR_E_INVAL, "record file: %s holds %lld pairs, not %lld", path,
                   (long long)h[0], (long long)n_pairs);
    }
    int64_t end = 0;
    emr_status st = scan(F->f, size, n_pairs, &end, &F->next, &F->records);
    if (st == EMR_OK && end < size && ::ftruncate(fileno(F->f), (off_t)end) != 0)
      st = failf(EMR_E_IO, "record file: cannot cut the partial block of %s: %s", path,
                 std::strerror(errno));
    if (st == EMR_OK && ::fseeko(F->f, (off_t)end, SEEK_SET) != 0)
      st = failf(EMR_E_IO, "record file: cannot seek in %s", path);
    if (st != EMR_OK) {
      std::fclose(F->f);
      delete F;
      return st;
    }
  } else {
    F->f = std::fopen(path, "w+b");
    if (!F->f) {
      delete F;
      return failf(EMR_E_IO, "record file: cannot create %s: %s", path, std::strerror(errno));
    }
    const int64_t h[3] = {n_pairs, 0, 0};
    if (std::fwrite(kMagic, 1, 8, F->f) != 8 || std::fwrite(h, 1, sizeof h, F->f) != sizeof h ||
        std::fflush(F->f) != 0) {
      std::fclose(F->f);
      delete F;
      return failf(EMR_E_IO, "record file: cannot write %s: %s", path, std::strerror(errno));
    }
  }
  F->buf.resize((size_t)(buffer_bytes ? buffer_bytes : kDefaultBuffer));
  std::setvbuf(F->f, F->buf.data(), _IOFBF, F->buf.size());
  if (cursor) *cursor = F->next;
  *out = F;
  return EMR_OK;
}

}  // namespace

extern "C" {

emr_status emr_record_file_open(const char* path, int64_t n_pairs, int32_t resume,
                                int64_t buffer_bytes, emr_record_file** out, int64_t* cursor) {
  return open_file(path, n_pairs, resume, buffer_bytes, out, cursor);
}

int32_t emr_record_file_sink(int64_t pair, int64_t chunk, const uint32_t* parent, const float* w4,
                             int64_t n_records, void* user) {
  auto* F = static_cast<emr_record_file*>(user);
  if (!F || !F->f) return 1;
  if (F->failed != EMR_OK) return 1;
  char b[256];
  if (pair < 0 || pair >= F->n_pairs || chunk < 0 || chunk > (INT64_MAX - pair) / F->n_pairs ||
      n_records < 1 || !parent || !w4) {
    std::snprintf(b, sizeof b, "record file: bad delivery (pair %lld of %lld, chunk %lld, %lld "
                  "records)", (long long)pair, (long long)F->n_pairs, (long long)chunk,
                  (long long)n_records);
    F->msg = b;
    F->failed = EMR_E_INVAL;
    return 1;
  }
  const int64_t c = chunk * F->n_pairs + pair;
  if (c < F->next) {
    std::snprintf(b, sizeof b, "record file: delivery cursor %lld precedes the file's next "
                  "cursor %lld (resume from the cursor the open call returned)", (long long)c,
                  (long long)F->next);
    F->msg = b;
    F->failed = EMR_E_INVAL;
    return 1;
  }
  const int64_t h[3] = {pair, chunk, n_records};
  const size_t n = (size_t)n_records;
  if (std::fwrite(h, 1, sizeof h, F->f) != sizeof h ||
      std::fwrite(parent, sizeof(uint32_t), n, F->f) != n ||
      std::fwrite(w4, 4 * sizeof(float), n, F->f) != n) {
    std::snprintf(b, sizeof b, "record file: write failed at cursor %lld: %s", (long long)c,
                  std::strerror(errno));
    F->msg = b;
    F->failed = EMR_E_IO;
    return 1;
  }
  F->next = c + 1;
  F->records += n_records;
  return 0;
}

emr_status emr_record_file_close(emr_record_file* F, int64_t* records, int64_t* next) {
  if (!F) return failf(EMR_E_INVAL, "record file: NULL handle");
  bool io_ok = std::fflush(F->f) == 0;
  io_ok = ::fsync(fileno(F->f)) == 0 && io_ok;
  const int err = errno;
  io_ok = std::fclose(F->f) == 0 && io_ok;
  if (records) *records = F->records;
  if (next) *next = F->next;
  std::string msg = F->msg;
  const emr_status failed = F->failed;
  delete F;
  if (failed != EMR_OK) return failf(failed, "%s", msg.c_str());
  if (!io_ok) return failf(EMR_E_IO, "record file: flush failed: %s", std::strerror(err));
  return EMR_OK;
}

}  // extern "C"
