// Internal tables shared by the library's host builder (api.cpp) and its
// device engine (engine.hip).  Not part of the public ABI.
#pragma once
#include <stdint.h>

namespace simgpu {

constexpr uint32_t kNever = 0xFFFFFFFFu;
// Largest cycle a run may process: completion = cycle + 1 and ready =
// cycle + latency must both fit in u32.
constexpr uint64_t kCycleLimit = 0xFFFFFFFEull - (1ull << 20);

// Per-scenario device status.
// kRunWatchdog: more processed cycles than any correct run can need (every
// processed cycle either moves a line or jumps to a strictly later FIFO-head
// ready time), i.e. an engine fault; it ends the kernel instead of spinning.
enum : int32_t { kRunOk = 0, kRunDeadlock = 7, kRunMaxCycles = 8, kRunWatchdog = 10, kRunInternal = 11, kRunRunning = -1 };

// Everything a kernel needs, passed by value as the kernel argument.
// "Static" tables are shared by all scenarios; "state" arrays have one slice
// per scenario (scenario-major).
struct DevNet {
    // sizes
    int32_t m;           // links
    int32_t n_fsrc;      // links that carry traffic (FIFO sources / targets)
    int32_t ns;          // injection streams
    int32_t nflows;      // flow slots (distinct (src, dst) pairs used)
    int32_t S;           // scenarios
    int32_t arb;         // 0 lowest id, 1 round-robin
    int32_t bmax;        // max bandwidth over links and scenarios
    int32_t fifo_total;  // FIFO entries per scenario
    int32_t req_total;   // request slots per scenario
    int64_t T;           // transactions per scenario
    uint64_t max_cycles; // simulated-cycle guard
    uint64_t watchdog;   // processed-cycle bound (see kRunWatchdog)

    // static topology tables
    const int32_t *fsrc_link;     // [n_fsrc] link ids carrying traffic
    const int32_t *port_at_head;  // [m] input-port index of l at head(l)
    const int32_t *nports_tail;   // [m] number of input ports at tail(l)
    const int32_t *fifo_off;      // [m] offset of l's ring in a scenario's FIFO storage
    const int32_t *fifo_mask;     // [m] ring size - 1 (power of two >= max cap)
    const int32_t *req_off;       // [m] offset of l's request slots
    // injection streams: lines with the same source and first link, in id order,
    // as a list of id ranges
    const int32_t *s_link;        // [ns] first link
    const int32_t *s_rbeg;        // [ns] first range
    const int32_t *s_rend;        // [ns] one past last range
    const uint32_t *r_start;      // [nr] first line id
    const uint32_t *r_len;        // [nr] lines in range
    const int32_t *r_path;        // [nr] index of the range's first hop in path_link
    const int32_t *r_pd;          // [nr+1] predecessor descriptors of the range
    // resident engine: the same descriptors with a range that repeats the
    // descriptors of the range before it in its stream sharing that range's
    // span (a group's stores all wait on the group's loads): range j's
    // descriptors are wr_pdf/wr_pdb[wr_rpb[j] .. wr_rpe[j] - 1]
    const int32_t *wr_rpb, *wr_rpe, *wr_pdf;
    const uint32_t *wr_pdb;
    // predecessor descriptor: line start+o may be injected once flow pd_flow has
    // delivered more than pd_base + (o & pd_omask) lines (flows deliver in id
    // order).  pd_omask is all ones for per-line dependencies; 0 for per-chunk
    // ones, where pd_base is the last line of the predecessor chunk.
    const int32_t *pd_flow;
    const uint32_t *pd_base;
    uint32_t pd_omask;
    // paths: hop link ids, each path terminated by -(1 + flow slot)
    const int32_t *path_link;
    // workgroup engine: streams that wait on a flow ([nflows+1] CSR), woken
    // when the flow delivers
    const int32_t *fw_ptr, *fw_str;

    // per-scenario parameters [S*m]
    const int32_t *bw, *lat, *cap;
    const int32_t *credit;  // [S*m] credit return delay, or null when every delay is 1
    const uint8_t *line_cls;  // [T] message class (1 control, 0 data) or null (all data)

    // per-scenario state
    uint32_t *fifo_x;     // [S*fifo_total] line id
    uint32_t *fifo_rdy;   // [S*fifo_total] first cycle the entry may leave
    int32_t *fifo_pp;     // [S*fifo_total] path index of the link the entry is on
    uint32_t *qhead;      // [S*m] popped count
    uint32_t *qtail;      // [S*m] pushed count
    uint32_t *cptr;       // [S*m] class-fair arbitration: the class that goes first
    int32_t wg_lds;       // workgroup engine: bytes of per-scenario scalars kept in LDS (0: in HBM)
    int32_t wg_act;       // workgroup engine: bytes of the active sets in LDS after them (0: full scans)
    int32_t wg_rcap;      // workgroup engine: capacity of the active sets' request list
    int32_t wg_scap;      // workgroup engine: capacity of the active sets' spill list (chunks of long FIFO offers)
    uint32_t *qcred;      // [S*m] popped entries whose slot is free again (credit returned);
                          // a popped entry's fifo_rdy then holds the cycle it left
    uint32_t *rr;         // [S*m] round-robin pointer
    int32_t *cur_rng;     // [S*ns] stream cursor: range
    uint32_t *cur_off;    // [S*ns] stream cursor: offset in range
    uint32_t *delivered;  // [S*nflows] lines delivered per flow

    // per-scenario scratch
    uint32_t *req_cnt;    // [S*m] requests received this cycle
    uint64_t *req_rec;    // [S*req_total] (key << 32) | (source << 8) | k
    uint32_t *req_aux;    // [S*req_total] class-fair picks: requests of the same source ahead
    uint32_t *sreq_x;     // [S*(m+ns)*bmax] requested line
    int32_t *sreq_pp;     // [S*(m+ns)*bmax] path index of the requested hop
    int32_t *sreq_n;      // [S*(m+ns)] requests made this cycle
    int32_t *grant;       // [S*(m+ns)*bmax] -1 none, -2 sink, else grant rank
    uint32_t *gcount;     // [S*m] grants issued this cycle
    uint32_t *glist;      // [S*m*bmax] (source << 8) | k by grant rank
    uint8_t *gdep;        // [S*m*bmax] granted request actually departs

    // lane engine: one lane per traffic-carrying link, a scenario's whole
    // state in one workgroup's LDS and registers
    int32_t engine;       // kEngineWorkgroup or kEngineLane
    int32_t nl;           // lanes (= n_fsrc), lane i owns link fsrc_link[i]
    int32_t lane_threads; // workgroup size of the lane engine (multiple of 64, >= nl)
    int32_t bm;           // compile-time bandwidth bound (power of two >= bmax)
    int32_t lds_bytes;    // dynamic LDS per workgroup
    int32_t o_path, o_deliv, o_reqcnt, o_reqb, o_req, o_glist, o_grant, o_gdep, o_red;  // LDS byte offsets
    int32_t path_len;     // entries of path_lane
    int32_t path_in_lds;  // path table copied into LDS
    int32_t req_slots;    // request slots in LDS
    const int32_t *ln_P;      // [nl] input ports at the tail of the lane's link
    const int32_t *ln_port;   // [nl] port index of the lane's link at its head
    const int32_t *ln_fifo;   // [nl] first LDS FIFO entry
    const int32_t *ln_mask;   // [nl] ring size - 1
    const int32_t *ln_req;    // [nl] first request slot of the lane as a target
    const int32_t *ln_reqcap; // [nl] request slots of the lane
    const int32_t *ln_srbeg;  // [nl] stream ranges of the lane's link (empty if none)
    const int32_t *ln_srend;
    const int32_t *link_lane; // [m] lane of a link, -1 if no traffic
    const int32_t *path_lane; // path table with link ids replaced by lanes
    const int32_t *ln_link;   // [nl] link of a lane
    uint4 *gfifo;             // [S*fifo_total] FIFO rings in HBM (lane-HBM and compact engines)

    // compact engine (every bandwidth 1): thread t owns lanes t, t+1024, ...
    int32_t has_preds;        // some line has predecessors
    int32_t b1_ns;            // stream lanes (lanes 0..b1_ns-1 start a stream)
    int32_t b1_lpt;           // lanes per thread
    int32_t b1_deliv_lds;     // delivered counters in LDS (required when lines have predecessors)
    int32_t o_word, o_gnt, o_inl, o_b1deliv, o_b1cnt, o_b1ino, o_b1red;  // LDS byte offsets
    int32_t b1_ring_lg;       // log2 of the (uniform) ring size
    const int32_t *in_lane;   // [m] lanes of each node's in-links in port order (-1: no traffic)
    const int32_t *ln_inoff;  // [nl] offset of the lane's tail node in in_lane

    // wave engine: G scenarios per wavefront, lane = (scenario slot, traffic link)
    int32_t wv_G;             // scenarios per wave (G * nl <= 64)
    int32_t wv_W;             // waves
    int32_t wv_nblk;          // workgroups: up to 16 independent waves each
    int32_t wv_wpb;           // wave slots per workgroup
    int32_t wv_nfs;           // request-slot groups per target lane: feeders + the lane's own stream
    int32_t wv_lineup;        // shift loop: a lane's feeder is lane - 1, its next link lane + 1
    const uint32_t *wv_duo;   // [nl] shift loop: local flows bound for the next lane (bit q)
    int32_t o_wword, o_wred, o_wdeliv, o_wreq, o_wgnt, o_wgdep;  // LDS byte offsets after a wave's rings
    const int32_t *blk_wave;  // [wv_nblk*wv_wpb] wave of each slot, -1 if empty
    const int32_t *blk_off;   // [wv_nblk*wv_wpb] LDS byte offset of the slot's region
    const int32_t *wv_sc;     // [wv_W*G] scenario of each slot, -1 if empty; longest expected runs first
    const uint32_t *wv_lfb;   // [nl] byte q: local flow q's next lane (the lane itself: leaves the network)
                              //   | its local index at the next lane << 6
    const uint32_t *wv_lfx;   // [nl] byte q: this lane's feeder index at local flow q's next lane
    const int32_t *pd_dix;    // [#descriptors] delivered-counter index of pd_flow: last lane * 4 + local index
    const int32_t *wv_feed;   // [nl*4] feeder lanes of a lane as a target: lane | port << 8
    const int32_t *wv_nfeed;  // [nl]
    const int32_t *r_lf;      // [nr] local flow index of a range's flow at its first lane

    // grid engine: one scenario, its nodes split over gd_nb workgroups that run
    // together; workgroup w is launched as block w * gd_stride
    int32_t gd_nb, gd_stride, gd_threads;
    int32_t gd_ns_max, gd_nt_max;  // most source / target sides of one workgroup
    int32_t gd_req_max;            // most request slots of one workgroup
    int32_t gd_fl_max;             // most delivered counters one workgroup keeps
    const int32_t *gd_sptr, *gd_slane;  // [gd_nb+1] CSR: lanes whose head node the workgroup owns
    const int32_t *gd_tptr, *gd_tlane;  // [gd_nb+1] CSR: lanes whose tail node the workgroup owns
    const int32_t *gd_rqoff;  // [nl] first request slot of a lane in its tail workgroup's slots
    const int32_t *gd_path;   // path table with hop lanes replaced by their index among the
                              //   tail workgroup's target sides (sink entries unchanged)
    const int32_t *gd_floc;   // [nflows] index of a flow's counter in its owner (-1: never waited on)
    const int32_t *gd_fptr, *gd_fown;  // [gd_nb+1] CSR: the flows each workgroup keeps counters of
    uint32_t *gd_pub;         // [4*nl] appended counts (cycle parity 0, 1), popped counts (0, 1)
    unsigned long long *gd_dslot;  // [2*nflows] delivered counts: (first cycle valid << 32) | count
    uint32_t *gd_sync;        // [16] arrival words [3 x 64 bit], next-cycle offers [3]
    // one-line-per-cycle form (every bandwidth 1; one source and one target
    // side per thread, in registers)
    int32_t gd_one;
    unsigned long long *gd_tpub;  // [2 parities x (appended, popped) x nl]: (cycle index << 32) | count
    // windowed form (every traffic link with latency and credit delay >= 2):
    // window length (0: not windowed), per-lane LDS ring offsets
    int32_t gd_window;
    int32_t gd_sring_max, gd_cring_max;  // most LDS ring entries of one workgroup's source / target sides
    const int32_t *gd_sro, *gd_tro;      // [nl] offset of a lane's mirrored entries / credit cycles
    int32_t gd_inl_max;       // most in-port table entries of one workgroup
    const int32_t *gd_toff;   // [nl] offset of a lane's tail node in its workgroup's in-port table
    const int32_t *gd_iptr, *gd_inl;  // [gd_nb+1] CSR: per node of the workgroup, for each input
                                      //   port the local source side feeding it (-1: stream or none)

    // resident workgroup engine: per-link state, link parameters and the
    // cycle's request records of a scenario in LDS (byte offsets wr_off),
    // records past wr_rcap in a per-scenario HBM overflow area of wr_ovf
    // entries per field
    int32_t wr_off[24];
    int32_t wr_rcap, wr_scap, wr_threads, wr_nw;  // wr_nw: windows of kResWindow ranges per stream
    int32_t wr_tcap;          // targets of a cycle whose per-target words are in LDS
    int64_t wr_ovf, wr_tovf;  // overflow entries per scenario: records, targets
    uint4 *wr_frec;           // [S*fifo_total] FIFO entries {line, ready, path index, 0}
    uint32_t *wr_ox, *wr_okey, *wr_ots, *wr_osidx, *wr_ogl;  // [S*wr_ovf] overflow records
    int32_t *wr_opp;
    uint16_t *wr_osrc, *wr_og, *wr_osrcid, *wr_oaux;
    unsigned long long *wr_otmask;  // [S*wr_tovf] overflow per-target words
    uint32_t *wr_otseg;
    uint16_t *wr_otq;

    // outputs
    uint32_t *completion; // [S*T]
    uint64_t *tx_lines;   // [S*m]
    uint64_t *busy;       // [S*m]
    uint32_t *makespan;   // [S]
    int32_t *status;      // [S] (kRunInternal: an LDS request slot overflowed)
    uint64_t *cycles;     // [S] processed cycles
};

enum : int32_t { kEngineWorkgroup = 0, kEngineLane = 1, kEngineLaneHbm = 2, kEngineB1 = 3, kEngineWave = 4,
                 kEngineGrid = 5, kEngineResident = 6 };
// Wave engine entry words: line id << kWaveXShift | local-flow index (0..3)
// << 5, the low five bits free for a request slot number (so line ids must
// be below 2^25 - 1).
constexpr int kWaveXShift = 7;
// Request-slot groups per target lane of the wave engine's general loop:
// feeders plus the lane's own stream, 2 or kWaveMaxNF.
constexpr int kWaveMaxNF = 4;
// Waves per wave-engine workgroup (two per SIMD: 256 registers each).
constexpr int kWaveMaxWpb = 8;
// Registers cache up to this many predecessor descriptors of a stream's range.
constexpr int kPredCache = 8;
// Resident workgroup engine: a stream's ranges are checked this many at a time
// (one thread per window).
constexpr int kResWindow = 4;

// Launch the engine for all scenarios on `stream`; returns a hipError_t value.
int launch_engine(const DevNet &d, void *stream);

}  // namespace simgpu

#include <hip/hip_runtime.h>

namespace simgpu {
// per-engine launchers (one translation unit each)
hipError_t launch_workgroup(const DevNet &d, hipStream_t st);
hipError_t launch_lane_any(const DevNet &d, hipStream_t st);
hipError_t launch_b1_any(const DevNet &d, hipStream_t st);
hipError_t launch_wave_any(const DevNet &d, hipStream_t st);
hipError_t launch_grid_any(const DevNet &d, hipStream_t st);
hipError_t launch_resident(const DevNet &d, hipStream_t st);

}  // namespace simgpu
