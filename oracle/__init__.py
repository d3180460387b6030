"""CPU oracle for the streamFFN routed-expert path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import anything from this package.  The
HIP library never calls it, and it shares no code with the library: no
kernels, headers, helpers, tables or pre/post-processing.  Its inputs come
from the seeded workload generator (which holds none of the method's
arithmetic) or from the tests themselves.

Modules (each function cites the passage of the paper it follows):

* ``fp8``     -- OCP e4m3fn decode/encode written from the format definition,
                 plus 1x128 activation block quantisation.
* ``mx``      -- OCP MX formats: E2M1 and E8M0 decode, packed MXFP4 weight
                 matrices, MXFP8 (E4M3) block quantisation (the paper's
                 MXFP4 expert precision, Section 4.1).
* ``routing`` -- per-batch expert histogram, exclusive scan, tile-aligned
                 offsets, stable permutation and inverse map (Appendix C,
                 "Grouped FFN invocations").
* ``policy``  -- streamFFN batch composition: launch threshold theta and the
                 final flush (Section 3.2, "Launch threshold"), plus the
                 synchronous (wait-for-all) and per-chunk baselines (Section
                 4.3, ablation).
* ``ffn``     -- the routed-expert output: expert FFN = GEMM, activation,
                 GEMM (Appendix C), each routed contribution weighted by its
                 routing coefficient exactly once and summed at the source
                 token (Appendix C, "Output return and combine").  float64.
* ``calibration`` -- launch threshold theta(rho) and the FFN latency model
                 F(N) from a throughput profile (Section 3.2).
* ``oewf``    -- the OEWF coordinator: Algorithm 1, the reassignment
                 admission test and the versioned commit (Section 3.3,
                 Appendix C, Appendix E).

Precision readings (the paper fixes none of them) are stated per function.
"""
