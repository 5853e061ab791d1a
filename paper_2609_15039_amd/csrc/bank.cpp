// Noise bank (Sec. "Precomputing the Mask and Noise Correction"): corrections
// C = eta W^T precomputed for a range of rows of one noise stream, kept in a file,
// loaded per batch and handed out once.  The masks themselves are not stored: the
// fused call regenerates eta from (seed, stream_id, row), so a bank holds only C.
//
// File layout (little-endian), BANK_HEADER bytes of header then rows x N float32:
//   0  char[8] "SPLTBANK"    8  uint32 version (1)     12 uint32 header bytes (128)
//   16 int64 K               24 int64 N                32 uint64 seed
//   40 uint64 stream_id      48 int32 mech             52 int32 prec
//   56 double sensitivity    64 double epsilon         72 int64 row0
//   80 int64 rows            88 int64 consumed         96..127 zero
// `consumed` is the single-use watermark: rows row0 .. row0 + consumed - 1 have been
// handed out and are never handed out again; it is written to the file (and synced)
// before the rows it covers are read.
#include <errno.h>
#include <fcntl.h>
#include <stdio.h>
#include <string.h>
#include <sys/file.h>
#include <sys/stat.h>
#include <unistd.h>

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <string>

#include "splitee.h"

namespace {

constexpr char BANK_MAGIC[8] = {'S', 'P', 'L', 'T', 'B', 'A', 'N', 'K'};
constexpr uint32_t BANK_VERSION = 1;
constexpr int64_t BANK_HEADER = 128;
constexpr int64_t BANK_CHUNK = 256;          // rows per correction launch when creating
constexpr int64_t BANK_MAX_DIM = int64_t(1) << 30;
constexpr off_t CONSUMED_OFFSET = 88;

#pragma pack(push, 1)
struct Header {
    char magic[8];
    uint32_t version;
    uint32_t header_bytes;
    int64_t K, N;
    uint64_t seed, stream_id;
    int32_t mech, prec;
    double sensitivity, epsilon;
    int64_t row0, rows, consumed;
    char reserved[32];
};
#pragma pack(pop)
static_assert(sizeof(Header) == BANK_HEADER, "bank header is 128 bytes");
static_assert(offsetof(Header, consumed) == CONSUMED_OFFSET, "watermark offset");

bool full_pwrite(int fd, const void* buf, size_t n, off_t off)
{
    const char* p = static_cast<const char*>(buf);
    while (n > 0) {
        const ssize_t w = pwrite(fd, p, n, off);
        if (w < 0 && errno == EINTR) continue;
        if (w <= 0) return false;
        p += w;
        n -= (size_t)w;
        off += w;
    }
    return true;
}

bool full_pread(int fd, void* buf, size_t n, off_t off)
{
    char* p = static_cast<char*>(buf);
    while (n > 0) {
        const ssize_t r = pread(fd, p, n, off);
        if (r < 0 && errno == EINTR) continue;
        if (r <= 0) return false;
        p += r;
        n -= (size_t)r;
        off += r;
    }
    return true;
}

bool valid_header(const Header& h, off_t file_bytes)
{
    if (memcmp(h.magic, BANK_MAGIC, 8) != 0 || h.version != BANK_VERSION || h.header_bytes != BANK_HEADER)
        return false;
    if (h.K < 0 || h.N <= 0 || h.K > BANK_MAX_DIM || h.N > BANK_MAX_DIM) return false;
    if (h.rows < 0 || h.consumed < 0 || h.consumed > h.rows || h.row0 < 0) return false;
    if (h.mech < SPLITEE_MECH_LAPLACE || h.mech > SPLITEE_MECH_NONE) return false;
    if (h.prec < SPLITEE_PREC_F32 || h.prec > SPLITEE_PREC_BF16X3) return false;
    if (!(h.epsilon > 0.0) || !std::isfinite(h.epsilon) || !(h.sensitivity >= 0.0) || !std::isfinite(h.sensitivity))
        return false;
    const double data = (double)h.rows * (double)h.N * 4.0;
    return (double)file_bytes == (double)BANK_HEADER + data;
}

}  // namespace

struct splitee_bank {
    int fd;
    Header h;
    float* staging;        // pinned host rows for device loads, kept until close
    size_t staging_bytes;
};

extern "C" {

int splitee_bank_path(const char* dir, int64_t K, int64_t N, uint64_t stream_id, char* out, size_t out_len)
{
    if (!dir || !out || K < 0 || N < 0) return SPLITEE_ERR_ARG;
    const int n = snprintf(out, out_len, "%s/bank-s%016llx-k%lld-n%lld.spb", dir, (unsigned long long)stream_id,
                           (long long)K, (long long)N);
    return n > 0 && (size_t)n < out_len ? SPLITEE_OK : SPLITEE_ERR_ARG;
}

size_t splitee_bank_workspace_bytes(int64_t K, int64_t N, int prec)
{
    if (prec != SPLITEE_PREC_F32 && prec != SPLITEE_PREC_BF16X3) return 0;  // the corrections' modes
    const size_t fused = splitee_fused_workspace_bytes(BANK_CHUNK, N, K, prec);
    if (fused == 0) return 0;
    return fused + (size_t)BANK_CHUNK * (size_t)N * 4;
}

int splitee_bank_create(const char* path, const void* W, int w_type, int64_t ldw, int64_t K, int64_t N, int mech,
                        double sensitivity, double epsilon, uint64_t seed, uint64_t stream_id, uint64_t row0,
                        int64_t rows, int prec, void* workspace, size_t workspace_bytes, void* stream)
{
    if (!path || rows < 0 || (int64_t)row0 < 0) return SPLITEE_ERR_ARG;
    if (N <= 0 || K < 0 || N > BANK_MAX_DIM || K > BANK_MAX_DIM || N % 4 != 0) return SPLITEE_ERR_SHAPE;
    // validate every argument of the correction before touching the file system
    const size_t fused = splitee_fused_workspace_bytes(BANK_CHUNK, N, K, prec);
    if (fused == 0) return prec == SPLITEE_PREC_F32 || prec == SPLITEE_PREC_BF16X3 ? SPLITEE_ERR_SHAPE
                                                                                   : SPLITEE_ERR_UNSUPPORTED;
    int rc = splitee_correction(nullptr, N, W, w_type, ldw, 0, N, K, mech, sensitivity, epsilon, seed, stream_id,
                                row0, prec, nullptr, 0, stream);
    if (rc) return rc;
    if (rows > 0 && !W) return SPLITEE_ERR_ARG;
    if (rows > 0 && (!workspace || workspace_bytes < splitee_bank_workspace_bytes(K, N, prec)))
        return SPLITEE_ERR_WORKSPACE;
    if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u)) return SPLITEE_ERR_ALIGN;

    const int fd = open(path, O_RDWR | O_CREAT | O_EXCL, 0600);
    if (fd < 0) return SPLITEE_ERR_IO;
    Header h{};
    // the header is written last: until then the file has no magic and does not open
    bool ok = full_pwrite(fd, &h, sizeof h, 0);
    float* host = nullptr;
    const int64_t chunk = std::min<int64_t>(BANK_CHUNK, std::max<int64_t>(rows, 1));
    if (ok && rows > 0 && hipHostMalloc((void**)&host, (size_t)chunk * N * 4, hipHostMallocDefault) != hipSuccess) {
        host = nullptr;
        rc = SPLITEE_ERR_HIP;
        ok = false;
    }
    char* base = static_cast<char*>(workspace);
    float* cdev = rows > 0 ? reinterpret_cast<float*>(base + fused) : nullptr;
    const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    for (int64_t r = 0; ok && r < rows; r += chunk) {
        const int64_t m = std::min(chunk, rows - r);
        rc = splitee_correction(cdev, N, W, w_type, ldw, m, N, K, mech, sensitivity, epsilon, seed, stream_id,
                                row0 + (uint64_t)r, prec, workspace, fused, stream);
        if (rc) { ok = false; break; }
        if (hipMemcpyAsync(host, cdev, (size_t)m * N * 4, hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            rc = SPLITEE_ERR_HIP;
            ok = false;
            break;
        }
        if (!full_pwrite(fd, host, (size_t)m * N * 4, BANK_HEADER + (off_t)r * N * 4)) {
            rc = SPLITEE_ERR_IO;
            ok = false;
        }
    }
    if (host) hipHostFree(host);
    if (ok) {
        memcpy(h.magic, BANK_MAGIC, 8);
        h.version = BANK_VERSION;
        h.header_bytes = BANK_HEADER;
        h.K = K;
        h.N = N;
        h.seed = seed;
        h.stream_id = stream_id;
        h.mech = mech;
        h.prec = prec;
        h.sensitivity = sensitivity;
        h.epsilon = epsilon;
        h.row0 = (int64_t)row0;
        h.rows = rows;
        h.consumed = 0;
        ok = fsync(fd) == 0 && full_pwrite(fd, &h, sizeof h, 0) && fsync(fd) == 0;
        if (!ok && rc == SPLITEE_OK) rc = SPLITEE_ERR_IO;
    }
    close(fd);
    if (!ok) {
        unlink(path);
        return rc ? rc : SPLITEE_ERR_IO;
    }
    return SPLITEE_OK;
}

int splitee_bank_open(const char* path, splitee_bank** bank)
{
    if (!path || !bank) return SPLITEE_ERR_ARG;
    *bank = nullptr;
    const int fd = open(path, O_RDWR);
    if (fd < 0) return SPLITEE_ERR_IO;
    // one handle per bank file at a time, across processes: the watermark has one writer
    if (flock(fd, LOCK_EX | LOCK_NB) != 0) {
        const int e = errno;
        close(fd);
        return e == EWOULDBLOCK ? SPLITEE_ERR_BUSY : SPLITEE_ERR_IO;
    }
    struct stat st;
    Header h;
    if (fstat(fd, &st) != 0 || !full_pread(fd, &h, sizeof h, 0)) {
        close(fd);
        return SPLITEE_ERR_FORMAT;
    }
    if (!valid_header(h, st.st_size)) {
        close(fd);
        return SPLITEE_ERR_FORMAT;
    }
    splitee_bank* b = new (std::nothrow) splitee_bank{fd, h, nullptr, 0};
    if (!b) {
        close(fd);
        return SPLITEE_ERR_IO;
    }
    *bank = b;
    return SPLITEE_OK;
}

int splitee_bank_info(const splitee_bank* bank, splitee_bank_info_t* info)
{
    if (!bank || !info) return SPLITEE_ERR_ARG;
    const Header& h = bank->h;
    info->K = h.K;
    info->N = h.N;
    info->seed = h.seed;
    info->stream_id = h.stream_id;
    info->mech = h.mech;
    info->prec = h.prec;
    info->sensitivity = h.sensitivity;
    info->epsilon = h.epsilon;
    info->row0 = h.row0;
    info->rows = h.rows;
    info->consumed = h.consumed;
    info->bytes_stored = BANK_HEADER + h.rows * h.N * 4;
    info->bytes_with_masks = BANK_HEADER + h.rows * (h.N + h.K) * 4;
    return SPLITEE_OK;
}

int splitee_bank_load(splitee_bank* bank, int64_t rows, float* C, int64_t ldc, int dst_device, int64_t* row0,
                      void* stream)
{
    if (!bank || !row0 || rows < 0) return SPLITEE_ERR_ARG;
    Header& h = bank->h;
    if (rows == 0) {
        *row0 = h.row0 + h.consumed;
        return SPLITEE_OK;
    }
    if (!C) return SPLITEE_ERR_ARG;
    if (ldc < h.N) return SPLITEE_ERR_SHAPE;
    if (rows > h.rows - h.consumed) return SPLITEE_ERR_EXHAUSTED;
    // take the rows first: the watermark reaches the file before any of them is read
    const int64_t first = h.consumed, taken = h.consumed + rows;
    if (!full_pwrite(bank->fd, &taken, sizeof taken, CONSUMED_OFFSET) || fsync(bank->fd) != 0)
        return SPLITEE_ERR_IO;
    h.consumed = taken;
    *row0 = h.row0 + first;
    const off_t src = BANK_HEADER + (off_t)first * h.N * 4;
    const size_t row_bytes = (size_t)h.N * 4;
    if (!dst_device) {
        if (ldc == h.N) return full_pread(bank->fd, C, (size_t)rows * row_bytes, src) ? SPLITEE_OK : SPLITEE_ERR_IO;
        for (int64_t r = 0; r < rows; ++r)
            if (!full_pread(bank->fd, C + r * ldc, row_bytes, src + (off_t)r * row_bytes)) return SPLITEE_ERR_IO;
        return SPLITEE_OK;
    }
    // device destination: through a pinned staging buffer, BANK_CHUNK rows at a time
    const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int64_t chunk = std::min<int64_t>(rows, BANK_CHUNK);
    if (bank->staging_bytes < (size_t)chunk * row_bytes) {
        if (bank->staging) hipHostFree(bank->staging);
        bank->staging = nullptr;
        bank->staging_bytes = 0;
        if (hipHostMalloc((void**)&bank->staging, (size_t)chunk * row_bytes, hipHostMallocDefault) != hipSuccess) {
            bank->staging = nullptr;
            return SPLITEE_ERR_HIP;
        }
        bank->staging_bytes = (size_t)chunk * row_bytes;
    }
    float* host = bank->staging;
    int rc = SPLITEE_OK;
    for (int64_t r = 0; r < rows && rc == SPLITEE_OK; r += chunk) {
        const int64_t m = std::min(chunk, rows - r);
        if (!full_pread(bank->fd, host, (size_t)m * row_bytes, src + (off_t)r * row_bytes)) {
            rc = SPLITEE_ERR_IO;
            break;
        }
        if (hipMemcpy2DAsync(C + r * ldc, (size_t)ldc * 4, host, row_bytes, row_bytes, (size_t)m,
                             hipMemcpyHostToDevice, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess)
            rc = SPLITEE_ERR_HIP;
    }
    return rc;
}

int splitee_bank_close(splitee_bank* bank)
{
    if (!bank) return SPLITEE_ERR_ARG;
    if (bank->staging) hipHostFree(bank->staging);
    const int rc = close(bank->fd) == 0 ? SPLITEE_OK : SPLITEE_ERR_IO;
    delete bank;
    return rc;
}

}  // extern "C"
