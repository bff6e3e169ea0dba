// Microbenchmarks of the gfx950 units the GauS kernels lean on: fp32 FMA
// issue rate, v_exp_f32 / v_rcp_f32 (transcendental) rate, the device
// library's erfcf and expf for comparison, HBM copy/write bandwidth and a
// random row-gather pattern.  Prints one line per measurement; the ratio of
// the FMA to the v_exp_f32 rate is the transcendental weight of the VALU cost
// model used for the roofline.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#include <vector>
#include <cmath>
#define CK(x) do{hipError_t e=(x); if(e!=hipSuccess){printf("HIP error %s at %d\n",hipGetErrorString(e),__LINE__); exit(1);}}while(0)

template<int OP>
__global__ void kt(float* out, int iters, float seed) {
  int gid = blockIdx.x*blockDim.x + threadIdx.x;
  float a0 = seed + gid*1e-7f, a1 = a0+0.1f, a2=a0+0.2f, a3=a0+0.3f;
  float a4=a0+0.4f,a5=a0+0.5f,a6=a0+0.6f,a7=a0+0.7f;
  for (int i = 0; i < iters; ++i) {
    if (OP==0) { // exp2
      a0=__builtin_amdgcn_exp2f(a0); a1=__builtin_amdgcn_exp2f(a1); a2=__builtin_amdgcn_exp2f(a2); a3=__builtin_amdgcn_exp2f(a3);
      a4=__builtin_amdgcn_exp2f(a4); a5=__builtin_amdgcn_exp2f(a5); a6=__builtin_amdgcn_exp2f(a6); a7=__builtin_amdgcn_exp2f(a7);
      a0*=-0.5f;a1*=-0.5f;a2*=-0.5f;a3*=-0.5f;a4*=-0.5f;a5*=-0.5f;a6*=-0.5f;a7*=-0.5f;
    } else if (OP==1) { // rcp
      a0=__builtin_amdgcn_rcpf(a0); a1=__builtin_amdgcn_rcpf(a1); a2=__builtin_amdgcn_rcpf(a2); a3=__builtin_amdgcn_rcpf(a3);
      a4=__builtin_amdgcn_rcpf(a4); a5=__builtin_amdgcn_rcpf(a5); a6=__builtin_amdgcn_rcpf(a6); a7=__builtin_amdgcn_rcpf(a7);
      a0+=1.f;a1+=1.f;a2+=1.f;a3+=1.f;a4+=1.f;a5+=1.f;a6+=1.f;a7+=1.f;
    } else if (OP==2) { // fma
      a0=fmaf(a0,0.999f,0.001f);a1=fmaf(a1,0.999f,0.001f);a2=fmaf(a2,0.999f,0.001f);a3=fmaf(a3,0.999f,0.001f);
      a4=fmaf(a4,0.999f,0.001f);a5=fmaf(a5,0.999f,0.001f);a6=fmaf(a6,0.999f,0.001f);a7=fmaf(a7,0.999f,0.001f);
      a0=fmaf(a0,0.999f,0.001f);a1=fmaf(a1,0.999f,0.001f);a2=fmaf(a2,0.999f,0.001f);a3=fmaf(a3,0.999f,0.001f);
      a4=fmaf(a4,0.999f,0.001f);a5=fmaf(a5,0.999f,0.001f);a6=fmaf(a6,0.999f,0.001f);a7=fmaf(a7,0.999f,0.001f);
    } else if (OP==3) { // erfcf (device library)
      a0=erfcf(a0)*3.f-1.f; a1=erfcf(a1)*3.f-1.f; a2=erfcf(a2)*3.f-1.f; a3=erfcf(a3)*3.f-1.f;
      a4=erfcf(a4)*3.f-1.f; a5=erfcf(a5)*3.f-1.f; a6=erfcf(a6)*3.f-1.f; a7=erfcf(a7)*3.f-1.f;
    } else if (OP==4) { // expf (device library)
      a0=expf(a0)-1.5f; a1=expf(a1)-1.5f; a2=expf(a2)-1.5f; a3=expf(a3)-1.5f;
      a4=expf(a4)-1.5f; a5=expf(a5)-1.5f; a6=expf(a6)-1.5f; a7=expf(a7)-1.5f;
    }
  }
  out[gid] = a0+a1+a2+a3+a4+a5+a6+a7;
}

__global__ void kcopy(const float4* __restrict__ a, float4* __restrict__ b, size_t n) {
  size_t i = (size_t)blockIdx.x*blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x*blockDim.x;
  for (; i < n; i += stride) b[i] = a[i];
}
__global__ void kwrite(float4* __restrict__ b, size_t n) {
  size_t i = (size_t)blockIdx.x*blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x*blockDim.x;
  for (; i < n; i += stride) b[i] = make_float4(1.f,2.f,3.f,4.f);
}
// each wave: one output row r; sums rows idx[r*4+0..3] of F (rows of D floats)
__global__ void kgather(const float* __restrict__ F, const int* __restrict__ idx, float* __restrict__ out, int nrows, int D) {
  int wave = (blockIdx.x*blockDim.x + threadIdx.x) >> 6;
  int lane = threadIdx.x & 63;
  if (wave >= nrows) return;
  int j0=idx[wave*4+0], j1=idx[wave*4+1], j2=idx[wave*4+2], j3=idx[wave*4+3];
  float acc = 0.f;
  for (int t = lane; t < D; t += 64) {
    acc += F[(size_t)j0*D+t] + F[(size_t)j1*D+t] + F[(size_t)j2*D+t] + F[(size_t)j3*D+t];
  }
  out[(size_t)wave*64+lane] = acc;
}

int main() {
  hipDeviceProp_t p; CK(hipGetDeviceProperties(&p, 0));
  printf("device %s arch %s CUs %d clock %d kHz L2 %d MB  mem %zu GB\n", p.name, p.gcnArchName, p.multiProcessorCount, p.clockRate, p.l2CacheSize>>20, p.totalGlobalMem>>30);
  hipEvent_t e0,e1; CK(hipEventCreate(&e0)); CK(hipEventCreate(&e1));
  int blocks = p.multiProcessorCount*16, threads=256; int n = blocks*threads;
  float* out; CK(hipMalloc(&out, n*sizeof(float)));
  const char* names[] = {"v_exp_f32","v_rcp_f32","v_fma_f32(x2)","erfcf","expf"};
  for (int op=0; op<5; ++op) {
    int iters = (op>=3)? 200 : 2000;
    for (int rep=0; rep<3; ++rep) {
      CK(hipEventRecord(e0));
      switch(op){case 0: kt<0><<<blocks,threads>>>(out,iters,0.3f);break; case 1: kt<1><<<blocks,threads>>>(out,iters,0.3f);break;
        case 2: kt<2><<<blocks,threads>>>(out,iters,0.3f);break; case 3: kt<3><<<blocks,threads>>>(out,iters,0.3f);break; case 4: kt<4><<<blocks,threads>>>(out,iters,0.3f);break;}
      CK(hipEventRecord(e1)); CK(hipEventSynchronize(e1));
      float ms; CK(hipEventElapsedTime(&ms,e0,e1));
      double cnt = (double)n*iters*8*(op==2?2:1);
      if (rep==2) printf("%-14s %.3f ms  %.3e evals/s  = %.3f evals/clk/CU\n", names[op], ms, cnt/(ms*1e-3), cnt/(ms*1e-3)/(p.multiProcessorCount*(double)p.clockRate*1e3));
    }
  }
  // HBM copy
  size_t bytes = (size_t)4<<30; size_t n4 = bytes/16;
  float4 *a,*b; CK(hipMalloc(&a,bytes)); CK(hipMalloc(&b,bytes));
  CK(hipMemset(a,0,bytes));
  for (int rep=0; rep<3; ++rep) {
    CK(hipEventRecord(e0)); kcopy<<<p.multiProcessorCount*32,256>>>(a,b,n4); CK(hipEventRecord(e1)); CK(hipEventSynchronize(e1));
    float ms; CK(hipEventElapsedTime(&ms,e0,e1)); if(rep==2) printf("copy 4GB: %.3f ms -> %.1f GB/s (r+w)\n", ms, 2.0*bytes/(ms*1e-3)/1e9);
  }
  for (int rep=0; rep<3; ++rep) {
    CK(hipEventRecord(e0)); kwrite<<<p.multiProcessorCount*32,256>>>(b,n4); CK(hipEventRecord(e1)); CK(hipEventSynchronize(e1));
    float ms; CK(hipEventElapsedTime(&ms,e0,e1)); if(rep==2) printf("write 4GB: %.3f ms -> %.1f GB/s\n", ms, 1.0*bytes/(ms*1e-3)/1e9);
  }
  // random gather: table of R rows x D floats, nrows outputs each summing 4 random rows
  for (int cfg=0; cfg<3; ++cfg) {
    int D = 4096; int R = (cfg==0)? 50000 : (cfg==1? 12500 : 2500); // 800MB / 200MB / 40MB tables
    int nrows = 50000;
    size_t tb = (size_t)R*D*4; if (tb > bytes) { printf("skip\n"); continue; }
    std::vector<int> h(nrows*4); srand(1); for (auto& v: h) v = rand()%R;
    int* di; CK(hipMalloc(&di, h.size()*4)); CK(hipMemcpy(di,h.data(),h.size()*4,hipMemcpyHostToDevice));
    float* go; CK(hipMalloc(&go,(size_t)nrows*64*4));
    int th=256; int bl=(nrows*64+th-1)/th;
    for (int rep=0; rep<3; ++rep) {
      CK(hipEventRecord(e0)); kgather<<<bl,th>>>((const float*)a,di,go,nrows,D); CK(hipEventRecord(e1)); CK(hipEventSynchronize(e1));
      float ms; CK(hipEventElapsedTime(&ms,e0,e1)); if(rep==2) printf("gather R=%d rows (table %.0f MB): %.3f ms -> %.1f GB/s delivered\n", R, tb/1e6, ms, (double)nrows*4*D*4/(ms*1e-3)/1e9);
    }
    CK(hipFree(di)); CK(hipFree(go));
  }
  printf("done\n");
  return 0;
}
