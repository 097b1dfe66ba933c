"""Layer shapes (C, M, Wx, Wy, K) whose plans split each stage's channels
over several waves of a workgroup (partial sums added through LDS), shared by
the GPU tests of that machinery and the CPU test that checks the planner
still chooses it for them."""

# several host threads at once, one stream each
THREADS = [(512, 512, 9, 9, 3), (256, 256, 30, 30, 3), (512, 512, 16, 16, 3),
           (128, 128, 60, 60, 5)]
# two streams at once
TWO_STREAMS = [(512, 512, 9, 9, 3), (512, 512, 16, 16, 3)]
# back to back on one stream, plans with and without the wave split mixed
# (at least three with)
REUSE = [(512, 512, 9, 9, 3), (256, 256, 30, 30, 3), (64, 96, 20, 20, 3),
         (512, 512, 9, 9, 3), (128, 128, 60, 60, 5), (256, 256, 28, 28, 1)]
