/*
 * tg.h -- C ABI of the MI355X patch-stitching library (libtg.so).
 *
 * Tangram (arXiv 2404.09267) batches variable-size RoI patches from many cameras
 * by stitching them, unresized, onto fixed-size canvases so that a detector sees one
 * fixed-shape batch (Sec. I; Sec. III-B; Sec. III-C, Patch-stitching Solver), and
 * its accuracy is scored per frame (Sec. V-D). This library is that data path:
 *
 *   tg_plan_pack   host:   place RoI rectangles on canvases (no HIP calls)
 *   tg_stitch      device: scatter uint8 RGB crops into fp16 NCHW canvases,
 *                          normalise per channel, fill the rest with the pad value
 *   tg_unstitch    device: map detector boxes from canvas back to frame pixels
 *
 * Conventions for every call:
 *  - Pixels: origin top-left, x right, y down; integer rectangles are half-open,
 *    [x, x+w) x [y, y+h).
 *  - Ownership: the caller owns every buffer. The library allocates no device memory
 *    and keeps no global state; tg_plan_pack frees its host temporaries before it
 *    returns.
 *  - Asynchrony: tg_stitch and tg_unstitch only enqueue work on `stream` (a
 *    hipStream_t; NULL is the default stream) and never synchronise. Inputs must stay
 *    valid, and outputs untouched, until the stream has passed the call.
 *  - Errors: every int-returning call returns TG_OK (0) or a negative TG_E_* code and
 *    never lets a C++ exception cross the ABI. A device call that returns an error
 *    has enqueued nothing.
 *  - Device buffers need only their natural alignment (4 bytes for int32/float, 2 for
 *    fp16); tg_stitch takes a faster path when `out` is 16-byte aligned and canvas_w
 *    is a multiple of 8.
 */
#ifndef TG_H
#define TG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A source rectangle: RoI/patch `i` is [x, x+w) x [y, y+h) of frame `frame`.
 * The paper's patch information carries the patch size (Sec. III-C, Alg. 2 input
 * P_i = {w_i, h_i, t_ddl_i}); the frame id and offset are what the cloud needs to
 * cut the pixels and to send detections back. 20 bytes. */
typedef struct {
  int32_t frame, x, y, w, h;
} tg_roi;

/* Where RoI i sits: canvas id and top-left corner on that canvas. Indexed like the
 * RoI table (the paper's assignment x_i^j, Sec. III-B). 12 bytes. */
typedef struct {
  int32_t canvas, x, y;
} tg_place;

/* A detector box in canvas pixels, continuous coordinates. 16 bytes. */
typedef struct {
  float x1, y1, x2, y2;
} tg_box;

/* A kept box mapped back to its frame: input box index, RoI index, frame id and the
 * box in frame pixels. 28 bytes. */
typedef struct {
  int32_t box, roi, frame;
  float x1, y1, x2, y2;
} tg_det;

enum tg_status {
  TG_OK = 0,
  TG_E_INVAL = -1,         /* null pointer, negative count, bad size/policy/std,
                              or an RoI with w < 1 or h < 1 */
  TG_E_ROI_TOO_LARGE = -2, /* RoI wider or taller than the canvas: patches are never
                              resized (Sec. III-C), so it cannot be placed */
  TG_E_ROI_OOB = -3,       /* RoI not inside its frame, or frame id out of range */
  TG_E_RANGE = -4,         /* canvas range outside [0, n_canvases) */
  TG_E_WORKSPACE = -5,     /* workspace missing or smaller than required */
  TG_E_HIP = -6,           /* the HIP runtime refused a launch */
  TG_E_INTERNAL = -7       /* host allocation failure or other internal error; also written
                              to a device count output when a device pass could not
                              complete (a grid-wide prefix whose predecessor never
                              published, a broken union-find link) */
};

enum tg_policy {
  /* First-fit decreasing height shelves: RoIs sorted by height, taller first (ties
   * keep input order); each goes on the first shelf of the current canvas that is
   * tall enough and has room, else on a new shelf under the last, else on a new
   * canvas. Closed canvases are not revisited. */
  TG_PACK_SHELF_FFDH = 0,
  /* The same shelves, RoIs taken in input (arrival) order. */
  TG_PACK_SHELF_ARRIVAL = 1,
  /* The paper's Patch-stitching Solver (Sec. III-C, Alg. 2): RoIs in input order;
   * among free rectangles that fit, the one leaving the smallest short-side leftover
   * min(w_c - w_i, h_c - h_i) (ties: smaller long-side leftover, then earlier in the
   * free list); the RoI goes to that rectangle's corner nearest the canvas origin;
   * the leftover is split in two along the free rectangle's shorter side; with no
   * fitting rectangle a new blank canvas is started. */
  TG_PACK_GUILLOTINE_BSSF = 2
};

typedef struct {
  int32_t canvas_w, canvas_h; /* canvas M x N of the paper (Sec. III-C), >= 1 */
  int32_t frame_w, frame_h;   /* every source frame's size, >= 1 */
  int32_t n_frames;           /* valid frame ids are [0, n_frames) */
  int32_t policy;             /* enum tg_policy */
} tg_pack_params;

/*
 * Pack n RoIs onto canvases of canvas_w x canvas_h (host only; makes no HIP call).
 *
 * Every RoI is placed exactly once, unrotated and unresized, with the rectangles on
 * one canvas pairwise disjoint and inside the canvas (Sec. III-B, constraints (3)
 * and (4); Sec. III-C). Canvases are opened one after another.
 *
 * In:  rois[n] (host). n >= 0.
 * Out (host, caller-allocated):
 *   place[n]            placement of RoI i
 *   order[n]            RoI ids in placement sequence; canvas-major
 *   canvas_begin[n+1]   order[canvas_begin[j] .. canvas_begin[j+1]) lie on canvas j;
 *                       entries 0 .. *n_canvases are written
 *   *n_canvases         J, the number of canvases (0 when n == 0)
 *   *bad_index          -1, or the first RoI that failed validation
 * RoIs are validated in index order; the first failure decides the code: w or h < 1
 * -> TG_E_INVAL; outside its frame or frame id not in [0, n_frames) -> TG_E_ROI_OOB;
 * larger than the canvas -> TG_E_ROI_TOO_LARGE. Outputs are unspecified on error.
 */
int tg_plan_pack(const tg_roi *rois, int32_t n, const tg_pack_params *params,
                 tg_place *place, int32_t *order, int32_t *canvas_begin,
                 int32_t *n_canvases, int32_t *bad_index);

/*
 * Batch split: the paper caps the canvases per function invocation by the GPU memory
 * one canvas takes (Sec. III-B, constraint (5)). Batch k holds canvases
 * [k * batch_cap, min((k+1) * batch_cap, n_canvases)); batch_cap <= 0 means one batch
 * holding every canvas.
 * tg_batch_count returns the number of batches (0 for no canvases).
 * tg_batch_range writes batch k's first canvas and count; TG_E_RANGE if k is not a
 * batch, TG_E_INVAL on null pointers.
 */
int32_t tg_batch_count(int32_t n_canvases, int32_t batch_cap);
int tg_batch_range(int32_t n_canvases, int32_t batch_cap, int32_t k, int32_t *first,
                   int32_t *count);

/*
 * Plan upload (data movement only, no step of the method): copies `bytes` from pinned
 * host memory `src` (hipHostMalloc, or a torch tensor made with pin_memory=True) to
 * device memory `dst` with one kernel on `stream` that reads `src` over PCIe -- for a
 * serving loop that hands each step's plan (tg_plan_pack's place, order, canvas_begin)
 * to the device. `src` must stay unchanged until the stream has passed the kernel; `dst`
 * belongs to the caller. Returns TG_OK (bytes == 0 enqueues nothing), TG_E_INVAL for a
 * null pointer or for `src` that is not pinned memory the device can read (checked with
 * hipHostGetDevicePointer before anything is enqueued), TG_E_HIP on launch failure.
 */
int tg_plan_upload(const void *src, void *dst, size_t bytes, void *stream);

/* ---- Adaptive frame partitioning (Sec. III-A, Alg. 1) ---- */

typedef struct {
  /* RoIs from the background model, device, grouped by frame: frame f's RoIs are
   * boxes[frame_begin[f] .. frame_begin[f+1]) and have .frame == f. */
  const tg_roi *boxes;
  const int32_t *frame_begin;  /* device [n_frames + 1] */
  int32_t n_boxes, n_frames, frame_w, frame_h;
  int32_t zones_x, zones_y;    /* X x Y zones, X <= frame_w, Y <= frame_h, X * Y <= 1024 */
  tg_roi *patches;             /* device out [n_boxes]: the first *n_patches are valid */
  int32_t *zone_of_box;        /* device out [n_boxes], or null: zone r* of each RoI, -1 if
                                  the RoI is skipped */
  int32_t *n_patches;          /* device out, one int32 */
  void *workspace;             /* device scratch, >= tg_partition_workspace_bytes(n_frames),
                                  8-byte aligned */
  size_t workspace_bytes;
} tg_partition_args;

/* Device scratch tg_partition needs for n_frames frames (0 when n_frames <= 0). */
size_t tg_partition_workspace_bytes(int32_t n_frames);

/*
 * Adaptive frame partitioning (Sec. III-A, Alg. 1): each frame is divided into
 * zones_x x zones_y zones; zone i of X spans columns [floor(i W / X), floor((i+1) W / X))
 * and zone j of Y rows [floor(j H / Y), floor((j+1) H / Y)); zone r = j * X + i. Every
 * RoI joins the zone with the largest overlap area (ties: the lowest r), and every zone
 * with RoIs becomes one patch, the minimum rectangle enclosing its RoIs (not clipped to
 * the zone). Patches are written frame by frame, zones in increasing r, as tg_roi records
 * (frame, x, y, w, h), ready for tg_plan_pack; a patch may be larger than a canvas, which
 * tg_plan_pack then reports. RoIs that are not inside the frame, have w or h < 1, or carry
 * another frame id are skipped (zone -1). Enqueued on `stream`; the library allocates
 * nothing. Returns TG_E_INVAL (null pointer, negative count, bad sizes, more than 1024
 * zones), TG_E_WORKSPACE, TG_E_HIP. With n_frames == 0 only *n_patches = 0 is written.
 */
int tg_partition(const tg_partition_args *args, void *stream);

/* ---- Online SLO-aware batching invoker (Sec. III-C, Alg. 2; Latency Estimator) ---- */

/* A patch as the scheduler receives it: its size, the time it arrives and its deadline
 * (generation time plus SLO). Times are in any one unit (seconds, say), finite. */
typedef struct {
  int32_t w, h;
  double t_arrive;
  double t_ddl;
} tg_slo_patch;

typedef struct {
  int32_t canvas_w, canvas_h;
  int32_t policy;          /* TG_PACK_GUILLOTINE_BSSF (the paper's solver) or
                              TG_PACK_SHELF_ARRIVAL: packers that keep arrival order */
  int32_t max_canvases;    /* memory cap: canvases one invocation may hold (>= 1) */
  int32_t n_lat;           /* rows of the latency table, >= max_canvases */
  const double *lat_mean;  /* host [n_lat]: mean inference time of b canvases at row b-1 */
  const double *lat_std;   /* host [n_lat]: its standard deviation */
} tg_slo_params;

enum tg_fire_reason {
  TG_FIRE_DEADLINE = 0, /* the clock reached t_remain = t_DDL - T_slack */
  TG_FIRE_SLO = 1,      /* the next patch would have pushed t_remain before its arrival */
  TG_FIRE_MEMORY = 2    /* the next patch would have needed more than max_canvases */
};

/* One invocation of the detector function. */
typedef struct {
  double t_fire;        /* when it is invoked */
  double t_ddl;         /* earliest deadline among its patches (t_DDL) */
  double t_slack;       /* Latency Estimator's conservative time for its batch */
  int32_t first, count; /* its patches: order[first .. first+count), in arrival order */
  int32_t n_canvases;
  int32_t reason;       /* enum tg_fire_reason */
} tg_invocation;

/*
 * Replays an arrival trace through the SLO-aware batching invoker of Alg. 2 (Sec. III-C):
 * on each arrival the patch joins the queue, t_DDL becomes the earliest deadline of the
 * queue, the queue is packed onto canvas_w x canvas_h canvases, the Latency Estimator
 * gives T_slack = lat_mean[b-1] + 3 * lat_std[b-1] for the b canvases, and
 * t_remain = t_DDL - T_slack. If t_remain falls before the arrival time, or b exceeds
 * max_canvases, the queue without the new patch is invoked at the arrival time and the
 * patch starts a new queue. Whenever the clock reaches t_remain (t >= t_remain), the queue
 * is invoked at max(t_remain, the time it was last changed); a deadline firing that falls
 * exactly on an arrival time happens before that arrival. After the last arrival the queue
 * fires at its t_remain. The paper's pseudo-code tests `t_remain > t` where its text
 * describes the opposite; this library reads it as stated above.
 * The queue is packed incrementally, one placement per arrival: with an arrival-order
 * packer that equals packing the whole queue afresh on every arrival, as Alg. 2 does.
 * patches: host [n], sorted by t_arrive (non-decreasing). Outputs (host, caller-owned):
 * order[n] (patch ids grouped by invocation), place[n] (indexed by patch id; canvas is
 * the canvas index inside its invocation), inv[n] (invocations, *n_inv of them).
 * Returns TG_E_INVAL (null pointer, n < 0, bad sizes or table, a policy that reorders,
 * a non-finite time, arrivals out of order: *bad_index names the patch when one is at
 * fault), TG_E_ROI_TOO_LARGE (patch larger than the canvas, *bad_index set),
 * TG_E_INTERNAL (host allocation failure).
 */
int tg_slo_replay(const tg_slo_patch *patches, int32_t n, const tg_slo_params *params,
                  int32_t *order, tg_place *place, tg_invocation *inv, int32_t *n_inv,
                  int32_t *bad_index);

typedef struct {
  /* Source frames, device, uint8 HWC RGB: pixel (x, y) of frame f, channel k, is
   * frames[f * frame_stride + y * row_pitch + 3 * x + k]. row_pitch >= 3 * frame_w,
   * frame_stride >= frame_h * row_pitch. */
  const uint8_t *frames;
  int64_t frame_stride;
  int32_t n_frames, frame_w, frame_h, row_pitch;
  /* The plan, device copies of tg_plan_pack's outputs for n_rois RoIs and
   * n_canvases canvases. */
  const tg_roi *rois;
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin; /* n_canvases + 1 entries */
  int32_t n_rois, n_canvases;
  /* Canvases [canvas_first, canvas_first + canvas_count) are written. */
  int32_t canvas_first, canvas_count;
  int32_t canvas_w, canvas_h;
  /* Per-channel normalisation in uint8 units, channels R, G, B: a source byte x of
   * channel k becomes binary16((x - mean[k]) / std[k]), the quotient taken in double
   * and rounded once to nearest-even binary16. std[k] must be finite and > 0, mean[k]
   * finite. Canvas pixels outside every patch get the same transform of pad[k]. */
  float mean[3], std[3];
  uint8_t pad[3];
  /* Output, device, binary16 bit patterns, [canvas_count][3][canvas_h][canvas_w]
   * contiguous: out[((c * 3 + k) * canvas_h + Y) * canvas_w + X] holds canvas
   * canvas_first + c. Every element is written exactly once. */
  uint16_t *out;
  /* Optional launch order of the work units, device, int32
   * [tg_stitch_units(canvas_w, canvas_h, canvas_count)]: workgroup b runs unit
   * unit_order[b]. NULL runs the units in id order, which is address order and the
   * fastest. The order changes only speed, never the output -- provided it is a
   * permutation: an id missing from it leaves that unit's pixels unwritten, a repeated
   * id writes them twice (same values), ids outside the range are ignored. */
  const int32_t *unit_order;
} tg_stitch_args;

/*
 * Stitch: for every canvas c in range, pixel (X, Y) and channel k, the output is the
 * normalised byte frames[f][Y - dy + sy][X - dx + sx][k] when (X, Y) lies in the
 * placed rectangle of an RoI on c (source (f, sx, sy), destination (dx, dy)), and the
 * normalised pad byte otherwise. The paper copies patches onto canvases without
 * resizing (Sec. I; Sec. III-C) but specifies no pixel mechanism; the transform above
 * is the detector input.
 *
 * The kernel trusts no plan entry: RoI ids outside [0, n_rois), RoIs whose place names
 * another canvas, and RoIs whose source or destination rectangle falls outside the
 * frame or canvas are skipped (their pixels read as pad), so a corrupt plan cannot make
 * it read or write outside the buffers described here.
 * Returns TG_E_INVAL for null pointers (unless canvas_count == 0), non-positive sizes,
 * row_pitch < 3 * frame_w, frame_stride < frame_h * row_pitch, or a bad mean/std;
 * TG_E_RANGE when the canvas range leaves [0, n_canvases); TG_E_HIP on launch failure.
 * canvas_count == 0 enqueues nothing and returns TG_OK.
 */
int tg_stitch(const tg_stitch_args *args, void *stream);

/*
 * Which exact normalisation tg_stitch uses for (mean, std) (host only): 0 when fp32
 * constants (a_k, c_k) exist with binary16(fma(x, a_k, c_k)) equal to the correctly
 * rounded binary16((x - mean[k]) / std[k]) for every byte x and channel k, so the kernel
 * computes each value; 1 when it looks values up in a 3 x 256 table instead. Both give
 * the same bits. TG_E_INVAL for null pointers or a bad mean/std (as tg_stitch).
 */
int32_t tg_stitch_norm_uses_table(const float mean[3], const float std[3]);

/*
 * Work units of one tg_stitch launch (host only). Each canvas plane is cut, in raster
 * order, into runs of 6144 pixels (the last run of a canvas may be shorter); one unit =
 * one run of one canvas, written in all three planes by one workgroup. Unit k is run
 * k % runs of canvas canvas_first + k / runs, with runs = ceil(canvas_w * canvas_h / 6144),
 * i.e. canvas pixels [6144 r, min(6144 (r + 1), canvas_w * canvas_h)).
 * Returns the number of units for canvas_count canvases of canvas_w x canvas_h (0 when
 * canvas_count == 0), or TG_E_INVAL for non-positive sizes, a negative count, or more
 * than 2^31 - 1 units.
 */
int32_t tg_stitch_units(int32_t canvas_w, int32_t canvas_h, int32_t canvas_count);

typedef struct {
  const tg_box *boxes;        /* device [n_boxes] */
  const int32_t *box_canvas;  /* device [n_boxes], canvas id of each box */
  int32_t n_boxes;
  const tg_roi *rois;         /* device plan, as for tg_stitch */
  const tg_place *place;
  const int32_t *order;
  const int32_t *canvas_begin;
  int32_t n_rois, n_canvases;
  int32_t clip;               /* nonzero: clip each kept box to its patch */
  int32_t *roi_of_box;        /* device out [n_boxes]: RoI id or -1 */
  tg_det *dets;               /* device out [n_boxes]: kept boxes, first *n_out valid */
  int32_t *n_out;             /* device out, one int32 */
  void *workspace;            /* device scratch, 16-byte aligned,
                                 >= tg_unstitch_workspace_bytes(n_boxes, n_rois) */
  size_t workspace_bytes;
  int32_t rule;               /* 0: the patch holding the box centre (default);
                                 1: the patch the box overlaps most, see tg_unstitch */
} tg_unstitch_args;

/*
 * Device scratch tg_unstitch needs for n_boxes boxes over a plan of n_rois RoIs (0 when
 * n_boxes <= 0): the compaction's look-back words (8 bytes per 1024 boxes and one more,
 * rounded up to 16) and 24 bytes of patch record per RoI.
 */
size_t tg_unstitch_workspace_bytes(int32_t n_boxes, int32_t n_rois);

/*
 * Unstitch: box b with canvas c = box_canvas[b]; its centre is
 * cx = (x1 + x2) * 0.5f, cy = (y1 + y2) * 0.5f in fp32 (no fused multiply-add).
 * It belongs to the RoI p on c with (float)dx <= cx < (float)(dx + w) and
 * (float)dy <= cy < (float)(dy + h) -- at most one, as placed rectangles are
 * disjoint. Boxes with no such RoI (centre on pad, NaN coordinate, or c outside
 * [0, n_canvases)) get roi_of_box[b] = -1 and are dropped. A kept box is clipped,
 * when `clip`, to [dx, dx+w] x [dy, dy+h] coordinate by coordinate (v < lo -> lo,
 * v > hi -> hi), then moved to frame pixels by adding (float)(sx - dx) to x1, x2 and
 * (float)(sy - dy) to y1, y2 (one fp32 add each). Kept boxes are written to dets in
 * increasing b (a stable compaction), and their count to *n_out. The paper scores
 * detections per frame (Sec. V-D) without stating this mapping; the centre rule is
 * this library's reading.
 * With rule = 1 a box instead belongs to the RoI p on c that it overlaps most: area =
 * ow * oh with ow = max(0, min(x2, dx+w) - max(x1, dx)) and oh likewise, binary32, one
 * rounding per operation; the largest area > 0 wins, ties go to the lower RoI id, and a
 * box with a NaN coordinate or no overlap is dropped (Alg. 1 assigns RoIs to zones by
 * largest overlap in the same way, Sec. III-A).
 * Returns TG_E_INVAL on null pointers (unless n_boxes == 0, which only writes
 * *n_out = 0) or n_boxes < 0, TG_E_WORKSPACE when the workspace is too small or not
 * 16-byte aligned, TG_E_HIP on launch failure, TG_E_INVAL for a rule other than 0 or 1.
 * *n_out = TG_E_INTERNAL reports a device-side failure of the compaction.
 */
int tg_unstitch(const tg_unstitch_args *args, void *stream);

/* Largest n_boxes tg_unstitch_noalloc accepts. */
#define TG_UNSTITCH_NOALLOC_MAX_BOXES (1 << 24)
/* Largest plan (n_rois) for which tg_unstitch_noalloc keeps patch records in its
 * scratch array; larger plans are read without them, with the same results. */
#define TG_UNSTITCH_NOALLOC_MAX_ROIS (1 << 17)

/*
 * tg_unstitch for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same operation and
 * results as tg_unstitch, but a->workspace and a->workspace_bytes are ignored. Instead the
 * call uses a scratch array the library holds in device memory, one per GPU: 3.3 MB that
 * each GPU the library runs on keeps until the process ends. The first call on a device
 * looks the array up (hipGetSymbolAddress); no call allocates or frees memory. The kernels
 * clear what they need themselves, so the array's contents from the previous call do not
 * matter -- but every call on one GPU shares it: calls that may overlap on one GPU (two
 * streams, two host threads) race and must be serialised by the caller.
 * Returns what tg_unstitch returns, except: TG_E_WORKSPACE when n_boxes >
 * TG_UNSTITCH_NOALLOC_MAX_BOXES; TG_E_HIP when the array cannot be looked up.
 */
int tg_unstitch_noalloc(const tg_unstitch_args *args, void *stream);

/* ---- Per-frame merge of detections after unstitch (Sec. III-A patches, Sec. V-D) ---- */

typedef struct {
  const tg_det *dets;       /* device [n_max]: tg_unstitch's output; box indices unique */
  const int32_t *n_dets;    /* device: how many of dets are valid (tg_unstitch's n_out) */
  int32_t n_max;            /* capacity of dets, keep and out */
  const float *scores;      /* device [n_scores]: detector score of each box, by tg_det.box */
  int32_t n_scores;
  int32_t n_frames;         /* frames are 0 .. n_frames-1 */
  float iou_threshold;
  int32_t cross_only;       /* nonzero: only detections from different patches suppress */
  int32_t *keep;            /* device out [n_max]: 1 kept, 0 dropped, for the first *n_dets */
  tg_det *out;              /* device out [n_max]: kept detections in input order */
  int32_t *n_kept;          /* device out, one int32 */
  void *workspace;          /* device scratch, >= tg_merge_workspace_bytes(n_max, n_frames),
                               16-byte aligned */
  size_t workspace_bytes;
} tg_merge_args;

/* Device scratch tg_merge needs (0 when n_max <= 0). */
size_t tg_merge_workspace_bytes(int32_t n_max, int32_t n_frames);

/*
 * Per-frame duplicate suppression of mapped-back detections. Patches of one frame can
 * overlap when a frame is cut into zone patches (Sec. III-A, Alg. 1), so one object can
 * come back twice; the paper scores per frame (Sec. V-D) without spelling out a merge.
 * This library's reading: a frame's detections are ranked by score (higher first; equal
 * scores by box index, lower first; a NaN score, or a box index outside [0, n_scores),
 * ranks as -infinity) and, walking the ranking, a detection is kept unless one kept
 * before it in the same frame (with cross_only: from another patch, tg_det.roi) overlaps
 * it by IoU > iou_threshold, decided in binary32 with every operation rounded on its own:
 * w = max(0, min(x2a, x2b) - max(x1a, x1b)), h likewise, inter = w * h,
 * area = max(0, x2 - x1) * max(0, y2 - y1), union = (area_a + area_b) - inter,
 * suppressed when inter > iou_threshold * union. Detections whose frame is outside
 * [0, n_frames) are dropped. Kept detections are written to out in input order and their
 * count to *n_kept. Every frame is merged, whatever its number of detections (the walk's
 * decisions are reached in parallel rounds over a spatial index of the frame's boxes,
 * kept in the workspace, with the same result). The
 * coordinates are not expected to be NaN (tg_unstitch never keeps such a box); if one is,
 * min and max ignore the NaN operand. Enqueued on `stream`; the library allocates nothing.
 * Returns TG_E_INVAL (null pointer, negative size, NaN threshold), TG_E_WORKSPACE,
 * TG_E_HIP. With n_max == 0 only *n_kept = 0 is written.
 * *n_kept = TG_E_INTERNAL reports a device-side failure (a compaction that could not
 * complete, or a frame whose rounds overran their bound; neither happens on a correct run).
 */
int tg_merge(const tg_merge_args *args, void *stream);

/* ---- Background model: the RoI source (Sec. III-A, step 1; Sec. V) ---- */

/* Most mixture components per pixel the kernels hold in registers. */
#define TG_GMM_MAX_MIX 5

typedef struct {
  int32_t n_mix;              /* K, components per pixel, 1 .. TG_GMM_MAX_MIX */
  float alpha;                /* learning rate of this frame, (0, 1] */
  float var_threshold;        /* background test: |x - mu|^2 < var_threshold * v */
  float var_threshold_gen;    /* ownership test: |x - mu|^2 < var_threshold_gen * v */
  float var_init;             /* variance of a new component, in [var_min, var_max] */
  float var_min, var_max;     /* 0 < var_min <= var_max */
  float background_ratio;     /* weight the background components cover (1 - c_f) */
  float complexity_reduction; /* c_T, in [0, 1) */
} tg_gmm_params;

typedef struct {
  const uint8_t *frames;  /* device [n_frames][height][width][3] RGB, packed, 4-byte aligned;
                             frame f is camera f's next sample */
  int32_t n_frames, width, height;
  float *state;           /* device, tg_gmm_state_bytes(n_px, n_mix) bytes, 16-byte aligned:
                             5 * n_mix planes of tg_gmm_plane_stride(n_px) floats, plane
                             5 m + {0: weight, 1..3: mean r, g, b, 4: variance} of
                             component m (heaviest first), pixel p = (f * height + y) *
                             width + x; only the first modes[p] components are meaningful */
  uint8_t *modes;         /* device [n_px], 4-byte aligned: components in use; all zero is a
                             fresh model (state contents are then ignored) */
  uint8_t *mask;          /* device out [n_px], 4-byte aligned: 1 foreground, 0 background */
  tg_gmm_params params;
} tg_gmm_args;

/* Floats between two state planes: n_px rounded up to a multiple of 64. */
int64_t tg_gmm_plane_stride(int64_t n_px);
/* Bytes of model state for n_px pixels and n_mix components (0 for bad arguments). */
size_t tg_gmm_state_bytes(int64_t n_px, int32_t n_mix);

/*
 * One frame per camera into each camera's per-pixel background model, n_px =
 * n_frames * width * height pixels. The paper takes its RoIs from a Gaussian-mixture
 * background model (Sec. III-A, step 1; Sec. V runs a MOG2-style subtractor); this is
 * the adaptive mixture whose component count is chosen online (Zivkovic, ICPR 2004),
 * with the background set of Stauffer and Grimson. Per pixel and sample x, in binary32
 * with every operation rounded on its own:
 *  1. components in order: d2 = |x - mu|^2 (r, g, b summed left to right); the first
 *     with d2 < var_threshold_gen * v owns x; x is background if a component whose
 *     predecessors' weights sum to at most background_ratio has d2 < var_threshold * v;
 *  2. w = (w + alpha (o - w)) - alpha c_T for every component (o = 1 for the owner); the
 *     owner, with rho = alpha / w: mu += rho (x - mu), v += rho (d2 - v), v clamped to
 *     [var_min, var_max];
 *  3. components with w < 0 are removed (the rest keep their order);
 *  4. with no owner a component (alpha, x, var_init) is appended, or replaces the last
 *     when n_mix are in use;
 *  5. weights are divided by their sum (list order); 6. stable sort, heaviest first.
 * mask[p] = 1 when x is not background. Enqueued on `stream`; allocates nothing.
 * Returns TG_E_INVAL (null pointer, non-positive sizes, misalignment, bad parameters),
 * TG_E_HIP. n_frames == 0 does nothing.
 */
int tg_gmm_update(const tg_gmm_args *args, void *stream);

typedef struct {
  const uint8_t *mask;      /* device [n_frames][height][width]: nonzero = foreground */
  int32_t n_frames, width, height;
  int32_t min_area;         /* components of fewer pixels are dropped */
  tg_roi *rois;             /* device out [max_rois]: bounding boxes {frame, x, y, w, h} */
  int32_t *areas;           /* device out [max_rois] or NULL: pixel count of each RoI */
  int32_t max_rois;
  int32_t *frame_begin;     /* device out [n_frames + 1]: RoIs of frame f are
                               [frame_begin[f], frame_begin[f + 1]) */
  int32_t *n_rois;          /* device out: kept components (more than max_rois: only the
                               first max_rois are written) */
  int32_t *n_components;    /* device out: all components; more than max_components means
                               the ones past the cap (raster order) were not measured */
  int32_t max_components;
  void *workspace;          /* device scratch, >= tg_mask_rois_workspace_bytes(...),
                               16-byte aligned */
  size_t workspace_bytes;
} tg_mask_rois_args;

/* Device scratch tg_mask_rois needs (0 for bad arguments). */
size_t tg_mask_rois_workspace_bytes(int32_t n_frames, int32_t width, int32_t height,
                                    int32_t max_components);

/*
 * RoIs from a foreground mask: the bounding boxes of each frame's 8-connected
 * foreground components of at least min_area pixels (the paper cuts its RoIs from the
 * background model's foreground, Sec. III-A, step 1; the connectivity, the area rule
 * and the order are this library's reading). RoIs are listed frame by frame, each
 * frame's in raster order of the component's first pixel, ready for tg_partition.
 * Enqueued on `stream`; allocates nothing. Returns TG_E_INVAL (null pointer,
 * non-positive sizes, more than 65535 frames or tile rows, width * height >= 2^30, 2^28 or
 * more 32x32 tiles over all frames, max_components < 1, max_rois < 0), TG_E_WORKSPACE,
 * TG_E_HIP. The workspace holds 4 bytes per pixel plus about 2.8 KB per 32x32 tile.
 * *n_rois = *n_components = TG_E_INTERNAL (no RoIs, frame_begin all 0) reports a
 * device-side failure: a union-find link that did not point to a smaller pixel index, or
 * a compaction that could not complete. Neither happens on a correct run; each loop that
 * could otherwise spin ends instead.
 */
int tg_mask_rois(const tg_mask_rois_args *args, void *stream);

/* Static description of a status code. */
const char *tg_strerror(int code);

/* ABI version: bumped whenever a struct or signature above changes. */
int32_t tg_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* TG_H */
