"""Layer shapes (C, M, Wx, Wy, K) whose plans split the channel sum across
workgroups, shared by the GPU tests of the split machinery and the CPU test
that checks the planner still splits them."""

# several host threads at once, one stream each
THREADS = [(512, 512, 9, 9, 3), (256, 256, 30, 30, 3), (512, 512, 16, 16, 3),
           (128, 128, 60, 60, 5)]
# two streams at once
TWO_STREAMS = [(512, 512, 9, 9, 3), (512, 512, 16, 16, 3)]
# back to back on one stream, split and unsplit plans mixed (at least three split)
REUSE = [(512, 512, 9, 9, 3), (256, 256, 30, 30, 3), (64, 96, 20, 20, 3),
         (512, 512, 9, 9, 3), (128, 128, 60, 60, 5), (256, 256, 28, 28, 1)]
