"""The workloads the hot path is measured and tested on.

Each pairs one GEMM ``K_g`` with one communication-side kernel ``K_c`` and is
run for ``n_iter`` GEMM -> collective iterations (Section 3.2, Fig. 1).  The
paper's own pairs (Table 1: cb-ar / mb-ar / cb-a2a / mb-a2a with 896 MB
collectives on 4-8 GPUs) become one GPU's local share of each collective:

* ``tiny``    -- GEMM 512^3 with a 4 x 2^20 float32 chunk sum;
* ``cb``      -- compute-bound GEMM 8192^3 (Table 1's cb shape) with an
                 8 x 2^25 float32 chunk sum;
* ``mb``      -- decode-like skinny GEMM 16 x 28672 x 8192 (weights N(0, 0.02))
                 with an 8 x 2^24 float32 chunk sum: both kernels are HBM-bound;
* ``a2a``     -- expert-like GEMM 16384 x 14336 x 4096 with a 64 x 4 MiB
                 chunk permutation (the local block of an alltoall);
* ``cb_own``  -- ``cb`` whose allreduce share consumes the GEMM's output:
                 iteration i's GEMM writes its own C_i and iteration i's
                 collective sums C_i (bf16, widened) and 7 fp32 peer chunks of
                 8192 x 8192 elements;
* ``sweep``   -- ``cb`` over extra LDS pads {0,16,32,64,96,128} KiB x comm wave
                 priority {normal, high};
* ``blocks``  -- ``cb`` with the paper's opt1 and opt2 tiles and a persistent
                 grid of X*X workgroups (the thread-block-count axis of
                 Figs. 2-3 and the tile-size study of Section 4.3);
* ``paper_*`` -- Table 1's own pairs on one GPU: cb (8192^3) and mb
                 (8192 x 57344 x 8192) GEMMs with an 896 MiB local share: a
                 4-chunk allreduce share (4 x 224 MiB fp32) or a 4-chunk
                 alltoall share (4 x 224 MiB).
"""
from dataclasses import dataclass, field

KIB = 1024
MIB = 1024 * 1024


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    comm: str                 # "reduce", "reduce_own" (first term: the GEMM's output) or "permute"
    nchunks: int
    length: int = 0           # float32 elements per chunk (reduce)
    chunk_bytes: int = 0      # bytes per chunk (permute)
    std_a: float = 1.0
    std_b: float = 1.0
    seed_b: int = None
    pads: tuple = (0,)
    priorities: tuple = (3,)
    n_iter: int = 10
    notes: str = field(default="", compare=False)

    @property
    def gemm_flops(self):
        return 2.0 * self.M * self.N * self.K

    @property
    def gemm_bytes(self):
        return 2.0 * (self.M * self.K + self.N * self.K + self.M * self.N)

    @property
    def comm_bytes(self):
        if self.comm == "reduce":
            return 4.0 * self.length * (self.nchunks + 1)
        if self.comm == "reduce_own":   # bf16 own term + nchunks fp32 peers + fp32 out
            return 2.0 * self.length + 4.0 * self.length * (self.nchunks + 1)
        return 2.0 * self.nchunks * self.chunk_bytes


WORKLOADS = {
    "tiny": Workload("tiny", 512, 512, 512, "reduce", 4, length=1 << 20,
                     pads=(0, 64 * KIB), priorities=(0, 3)),
    "cb": Workload("cb", 8192, 8192, 8192, "reduce", 8, length=1 << 25,
                   priorities=(0, 3)),
    "mb": Workload("mb", 16, 28672, 8192, "reduce", 8, length=1 << 24,
                   std_b=0.02, seed_b=4, priorities=(0, 3)),
    "a2a": Workload("a2a", 16384, 14336, 4096, "permute", 64, chunk_bytes=4 * MIB,
                    priorities=(0, 3)),
    "cb_own": Workload("cb_own", 8192, 8192, 8192, "reduce_own", 7, length=8192 * 8192,
                       priorities=(0, 3)),
    "sweep": Workload("sweep", 8192, 8192, 8192, "reduce", 8, length=1 << 25,
                      pads=tuple(p * KIB for p in (0, 16, 32, 64, 96, 128)),
                      priorities=(0, 3)),
    # the paper's thread-block-count axis (Figs. 2-3) and tile-size study
    # (Section 4.3): cb with the opt1 / opt2 tiles and a persistent grid of X*X
    # workgroups
    "blocks": Workload("blocks", 8192, 8192, 8192, "reduce", 8, length=1 << 25,
                       priorities=(0, 3)),
}
BLOCK_COUNTS = (8, 16, 32, 64, 128)   # X = Y; grid = X*X workgroups

# Table 1's workloads: 896 MiB collectives, P = 4 chunks of 224 MiB.
_SHARE = 224 * MIB
WORKLOADS.update({
    "paper_cb_ar": Workload("paper_cb_ar", 8192, 8192, 8192, "reduce", 4, length=_SHARE // 4,
                            priorities=(0, 3)),
    "paper_mb_ar": Workload("paper_mb_ar", 8192, 57344, 8192, "reduce", 4, length=_SHARE // 4,
                            priorities=(0, 3)),
    "paper_cb_a2a": Workload("paper_cb_a2a", 8192, 8192, 8192, "permute", 4, chunk_bytes=_SHARE,
                             priorities=(0, 3)),
    "paper_mb_a2a": Workload("paper_mb_a2a", 8192, 57344, 8192, "permute", 4, chunk_bytes=_SHARE,
                             priorities=(0, 3)),
})
