// Asynchronous post-processing of finished hypotheses (Section 4.3): while
// the GPU generates batch i + 1, a host thread turns the token ids of batch
// i into text and writes it out, so that detokenisation and output never
// hold up generation.
//
// A submitted batch is copied from device memory into one of `slots` staging
// buffers of pinned host memory by an asynchronous copy on the caller's
// stream, followed by an event; the worker thread waits for that event,
// detokenises the rows in order and appends one line per row.  Submission
// returns at once unless every staging buffer is still in use.
//
// Detokenisation is the byte-level decoding of the usual BPE vocabularies:
// each token id maps to a string of symbols, one symbol per byte, and the
// bytes are recovered symbol by symbol.  A byte that is a printable
// character stands for itself (0x21-0x7E, 0xA1-0xAC, 0xAE-0xFF); the other
// bytes, in increasing order, are written as the code points 0x100, 0x101, ...
// Symbols arrive as UTF-8; a row ends at its first end-of-sequence id or at
// its length, and ids outside the vocabulary are skipped.
#include <hip/hip_runtime.h>

#include <chrono>
#include <condition_variable>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <deque>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "fastseq_hip.h"
#include "launch.h"

namespace {

// code point -> byte of the byte-level alphabet (-1: not a symbol)
struct SymbolTable {
    int16_t byte_of[0x200];
    SymbolTable() {
        for (int c = 0; c < 0x200; ++c) byte_of[c] = -1;
        int extra = 0;
        for (int b = 0; b < 256; ++b) {
            const bool printable = (b >= 0x21 && b <= 0x7E) || (b >= 0xA1 && b <= 0xAC) || (b >= 0xAE && b <= 0xFF);
            if (printable) byte_of[b] = (int16_t)b;
            else byte_of[0x100 + extra++] = (int16_t)b;
        }
    }
};
const SymbolTable kSymbols;

struct Job {
    int slot, rows, t;
};

}  // namespace

struct fs_postproc {
    // vocabulary: token v is the UTF-8 text vocab[off[v] .. off[v+1])
    std::vector<char> vocab;
    std::vector<int64_t> off;
    int V = 0, eos = -1, max_rows = 0, max_len = 0, slots = 0;
    int32_t *staging = nullptr;           // pinned: slots x max_rows x max_len ids
    std::vector<hipEvent_t> copied;       // per slot: the batch's copy has landed
    std::FILE *file = nullptr;            // output file, or null: keep the bytes in `text`
    std::string text;
    // worker state
    std::mutex mu;
    std::condition_variable cv_job, cv_slot;
    std::deque<Job> jobs;
    std::vector<bool> busy;               // slot holds a batch not yet written
    int next_slot = 0, pending = 0;
    bool stop = false;
    int error = FS_OK;                    // first failure of the worker
    std::string error_text;
    double busy_seconds = 0.0;
    std::thread worker;

    // Appends the text of one row to `out`.
    void detokenize_row(const int32_t *ids, int t, std::string &out) const {
        for (int j = 0; j < t; ++j) {
            const int32_t v = ids[j];
            if (v == eos) break;
            if (v < 0 || v >= V) continue;
            const unsigned char *p = reinterpret_cast<const unsigned char *>(vocab.data() + off[v]);
            const unsigned char *e = reinterpret_cast<const unsigned char *>(vocab.data() + off[v + 1]);
            while (p < e) {
                int cp;
                if (p[0] < 0x80) {
                    cp = p[0];
                    p += 1;
                } else if ((p[0] & 0xE0) == 0xC0 && p + 1 < e) {
                    cp = ((p[0] & 0x1F) << 6) | (p[1] & 0x3F);
                    p += 2;
                } else {  // not a symbol of the alphabet: skip one byte
                    p += 1;
                    continue;
                }
                if (cp < 0x200 && kSymbols.byte_of[cp] >= 0) out.push_back((char)kSymbols.byte_of[cp]);
            }
        }
        out.push_back('\n');
    }

    void run() {
        std::string buf;
        for (;;) {
            Job job;
            {
                std::unique_lock<std::mutex> lock(mu);
                cv_job.wait(lock, [&] { return stop || !jobs.empty(); });
                if (jobs.empty()) return;  // stop requested and nothing left
                job = jobs.front();
                jobs.pop_front();
            }
            const hipError_t e = hipEventSynchronize(copied[job.slot]);
            const auto t0 = std::chrono::steady_clock::now();
            buf.clear();
            if (e == hipSuccess) {
                const int32_t *base = staging + (size_t)job.slot * max_rows * max_len;
                for (int r = 0; r < job.rows; ++r) detokenize_row(base + (size_t)r * job.t, job.t, buf);
            }
            {
                std::lock_guard<std::mutex> lock(mu);
                if (e != hipSuccess && error == FS_OK) {
                    error = FS_ERR_HIP;
                    error_text = std::string("post-process copy: ") + hipGetErrorString(e);
                }
            }
            if (e == hipSuccess) {
                if (file) {
                    if (std::fwrite(buf.data(), 1, buf.size(), file) != buf.size()) {
                        std::lock_guard<std::mutex> lock(mu);
                        if (error == FS_OK) {
                            error = FS_ERR_INVALID_ARG;
                            error_text = "post-process: write to the output file failed";
                        }
                    }
                } else {
                    text.append(buf);   // only the worker writes `text` before a flush
                }
            }
            const double dt = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
            {
                std::lock_guard<std::mutex> lock(mu);
                busy_seconds += dt;
                busy[job.slot] = false;
                --pending;
            }
            cv_slot.notify_all();
        }
    }
};

namespace {
int pp_fail(int status, const std::string &msg) { return fs::set_error(status, msg.c_str()); }
}  // namespace

extern "C" {

int fs_postproc_create(fs_postproc **out, const char *vocab, const int64_t *offsets, int V, int eos, int max_rows,
                       int max_len, int slots, const char *path)
{
    fs::set_error(FS_OK, "");
    if (!out) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_create: null output pointer");
    *out = nullptr;
    if (V < 1 || !vocab || !offsets) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_create: empty vocabulary");
    if (max_rows < 1 || max_len < 1 || slots < 1)
        return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_create: max_rows, max_len and slots must be >= 1");
    if ((long long)slots * max_rows * max_len > (1LL << 31))
        return pp_fail(FS_ERR_UNSUPPORTED, "fs_postproc_create: staging of more than 2^31 ids");
    if (offsets[0] != 0) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_create: offsets[0] must be 0");
    for (int v = 0; v < V; ++v)
        if (offsets[v + 1] < offsets[v])
            return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_create: offsets must not decrease");
    auto *pp = new fs_postproc();
    pp->vocab.assign(vocab, vocab + offsets[V]);
    pp->off.assign(offsets, offsets + V + 1);
    pp->V = V;
    pp->eos = eos;
    pp->max_rows = max_rows;
    pp->max_len = max_len;
    pp->slots = slots;
    pp->busy.assign(slots, false);
    if (path) {
        pp->file = std::fopen(path, "wb");
        if (!pp->file) {
            delete pp;
            return pp_fail(FS_ERR_INVALID_ARG, std::string("fs_postproc_create: cannot open ") + path);
        }
    }
    hipError_t e = hipHostMalloc(reinterpret_cast<void **>(&pp->staging),
                                 (size_t)slots * max_rows * max_len * sizeof(int32_t), hipHostMallocDefault);
    for (int s = 0; e == hipSuccess && s < slots; ++s) {
        hipEvent_t ev;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e == hipSuccess) pp->copied.push_back(ev);
    }
    if (e != hipSuccess) {
        for (hipEvent_t ev : pp->copied) (void)hipEventDestroy(ev);
        if (pp->staging) (void)hipHostFree(pp->staging);
        if (pp->file) std::fclose(pp->file);
        delete pp;
        return pp_fail(FS_ERR_HIP, std::string("fs_postproc_create: ") + hipGetErrorString(e));
    }
    pp->worker = std::thread([pp] { pp->run(); });
    *out = pp;
    return FS_OK;
}

int fs_postproc_submit(fs_postproc *pp, const int32_t *tokens, int ld, int rows, int t, void *stream)
{
    fs::set_error(FS_OK, "");
    if (!pp) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_submit: null handle");
    if (rows < 0 || t < 0 || ld < t) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_submit: bad sizes");
    if (rows > pp->max_rows || t > pp->max_len)
        return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_submit: batch larger than the staging buffers");
    if (rows > 0 && t > 0 && !tokens) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_submit: null tokens");
    int slot;
    {
        std::unique_lock<std::mutex> lock(pp->mu);
        if (pp->error != FS_OK) return pp_fail(pp->error, pp->error_text);
        slot = pp->next_slot;
        pp->cv_slot.wait(lock, [&] { return !pp->busy[slot]; });   // back-pressure: the slot's batch is written
        pp->busy[slot] = true;
        pp->next_slot = (slot + 1) % pp->slots;
        ++pp->pending;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int32_t *dst = pp->staging + (size_t)slot * pp->max_rows * pp->max_len;
    hipError_t e = hipSuccess;
    if (rows > 0 && t > 0)
        e = hipMemcpy2DAsync(dst, (size_t)t * 4, tokens, (size_t)ld * 4, (size_t)t * 4, rows, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipEventRecord(pp->copied[slot], s);
    if (e != hipSuccess) {
        std::lock_guard<std::mutex> lock(pp->mu);
        pp->busy[slot] = false;
        --pp->pending;
        pp->cv_slot.notify_all();
        return pp_fail(FS_ERR_HIP, std::string("fs_postproc_submit: ") + hipGetErrorString(e));
    }
    {
        std::lock_guard<std::mutex> lock(pp->mu);
        pp->jobs.push_back(Job{slot, rows, t});
    }
    pp->cv_job.notify_one();
    return FS_OK;
}

int fs_postproc_flush(fs_postproc *pp)
{
    fs::set_error(FS_OK, "");
    if (!pp) return pp_fail(FS_ERR_INVALID_ARG, "fs_postproc_flush: null handle");
    std::unique_lock<std::mutex> lock(pp->mu);
    pp->cv_slot.wait(lock, [&] { return pp->pending == 0; });
    if (pp->file && std::fflush(pp->file) != 0 && pp->error == FS_OK) {
        pp->error = FS_ERR_INVALID_ARG;
        pp->error_text = "post-process: flush of the output file failed";
    }
    if (pp->error != FS_OK) return pp_fail(pp->error, pp->error_text);
    return FS_OK;
}

size_t fs_postproc_output(fs_postproc *pp, char *buf, size_t cap)
{
    if (!pp) return 0;
    std::lock_guard<std::mutex> lock(pp->mu);
    if (pp->pending != 0) return 0;   // only between a flush and the next submit
    if (buf && cap) std::memcpy(buf, pp->text.data(), pp->text.size() < cap ? pp->text.size() : cap);
    return pp->text.size();
}

double fs_postproc_busy_seconds(fs_postproc *pp)
{
    if (!pp) return 0.0;
    std::lock_guard<std::mutex> lock(pp->mu);
    return pp->busy_seconds;
}

void fs_postproc_destroy(fs_postproc *pp)
{
    if (!pp) return;
    {
        std::lock_guard<std::mutex> lock(pp->mu);
        pp->stop = true;
    }
    pp->cv_job.notify_all();
    if (pp->worker.joinable()) pp->worker.join();
    for (hipEvent_t ev : pp->copied) (void)hipEventDestroy(ev);
    if (pp->staging) (void)hipHostFree(pp->staging);
    if (pp->file) std::fclose(pp->file);
    delete pp;
}

}  // extern "C"
