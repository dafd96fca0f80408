"""CPU oracle for the Fast Crossbar Model (FCM) evaluation path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 restatement of
what the method computes, written from the paper (RxNN, arXiv 1809.00072,
Sections III-VI).  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with the
HIP library under ``paper_1809_00072_amd/``, and it never imports that package.

Modules
-------
network   G -> G' (the non-ideal conductance matrix of one crossbar), twice:
          * ``gprime_nodal``: Kirchhoff current law at every node of the
            resistive network, solved with a library sparse LU.  This is the
            plain definition of the quantity the paper calls exact (Sec. V-A,
            generator step 3).
          * ``gprime_paper``: the paper's own six-step derivation
            (Sec. V-B, Eqs. 2-14), dense, with the sign reading documented there.
mapping   W -> tiles -> G per array -> G' (Sec. V-A, generator steps 1-3).
periph    DAC and ADC transfer models (Sec. IV-A, V-A; the curves themselves are
          a documented reading because the paper's figure is not available).
fcm       The evaluation phase: DAC, V.G' per tile (Eq. 14), ADC, digital
          accumulation across tiles, and conv-as-GEMM (Sec. VI).
variation Per-device variation factors (Philox-4x64-10 + Box-Muller) and the
          device characteristic table of generator step 2 (Sec. V-A).
backward  The floating-point backward pass of model-in-the-loop re-training
          (Sec. VI, its re-training paragraph), fully connected and convolution
          layers.

Parity status per function is stated in each module header.
"""
